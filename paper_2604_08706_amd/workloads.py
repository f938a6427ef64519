"""Seeded synthetic workloads shaped like the paper's replay batches.

This module only draws random inputs (shapes, value distributions, length mix,
reward rates).  It holds none of the method's arithmetic: no advantages, no
log-probabilities, no sampling rule.  Tests and the benchmark feed the same
draws to the HIP library and to the CPU oracle.

Workloads (stand-ins for the paper's OpenR1-Math-220k / MATH rollouts, which
are not available; rollout lengths log-normal, rewards Bernoulli, LM-head
weights and hidden states Gaussian):

* ``tiny``     d=64,   V=1024;   64 records (16 prompts x G=4), lengths U{8..32},
               8 draws padded to 32; staleness noise N(0, 0.05^2); rewards Bern(0.5).
* ``head05b``  d=896,  V=151936; 4096 records (512 x G=8), lengths LogN(ln 400, 0.5)
               capped at 1024; 64 uniform draws; noise N(0, 0.1^2); Bern(0.3).
* ``head15b``  d=1536, V=151936; 32768 records (4096 x G=8), LogN(ln 800, 0.5) cap
               4096; 512 draws, positive mixture p_pos = 0.7; policy age U{0..4} with
               noise sd 0.05 * age; Bern(0.3).
* ``head7b``   d=3584, V=152064; 1024 records (128 x G=8), LogN(ln 1200, 0.5) cap
               4096; 24 uniform draws, whose stream's first 16384 tokens form the
               micro-batch (enough draws that it is always full); noise N(0, 0.1^2);
               Bern(0.4).
* ``stress``   d=3584, V=152064; 10^6 records, LogN(ln 1200, 1.0) cap 8192; 256 draws,
               positive mixture p_pos = 0.5, padded; age U{0..4}; Bern(0.4).

Hidden states are N(0, 1) and W is N(0, 0.02^2) (bf16) unless a test asks
for peaked logits (larger W scale).  Token ids are uniform over the vocabulary.
"""

from dataclasses import dataclass

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    d: int
    V: int
    n_records: int
    group: int
    n_draw: int
    len_kind: str          # "uniform" or "lognormal"
    len_a: float           # uniform: low;  lognormal: median
    len_b: float           # uniform: high; lognormal: sigma
    len_cap: int
    reward_p: float
    noise_sd: float        # staleness noise of stored log-probs (per unit age if aged)
    aged: bool             # noise sd = noise_sd * age, age ~ U{0..4}
    mode: str              # "uniform" | "pos_mix" | "pos_retain"
    p_pos: float
    layout: str            # "packed" | "padded"
    max_tokens: int        # packed micro-batch size
    l_max: int             # padded row length


WORKLOADS = {
    "tiny": Workload("tiny", 64, 1024, 64, 4, 8, "uniform", 8, 32, 32, 0.5, 0.05, False,
                     "uniform", 0.0, "padded", 0, 32),
    "head05b": Workload("head05b", 896, 151936, 4096, 8, 64, "lognormal", 400, 0.5, 1024,
                        0.3, 0.1, False, "uniform", 0.0, "packed", 16384, 0),
    "head15b": Workload("head15b", 1536, 151936, 32768, 8, 512, "lognormal", 800, 0.5, 4096,
                        0.3, 0.05, True, "pos_mix", 0.7, "packed", 16384, 0),
    "head7b": Workload("head7b", 3584, 152064, 1024, 8, 24, "lognormal", 1200, 0.5, 4096,
                       0.4, 0.1, False, "uniform", 0.0, "packed", 16384, 0),
    "stress": Workload("stress", 3584, 152064, 1_000_000, 8, 256, "lognormal", 1200, 1.0, 8192,
                       0.4, 0.05, True, "pos_mix", 0.5, "padded", 0, 8192),
}


def lengths(wl, n, rng):
    """Rollout lengths: uniform integers or rounded log-normal, clamped to [1, cap]."""
    if wl.len_kind == "uniform":
        return rng.integers(int(wl.len_a), int(wl.len_b) + 1, n).astype(np.int64)
    x = np.rint(rng.lognormal(np.log(wl.len_a), wl.len_b, n))
    return np.clip(x, 1, wl.len_cap).astype(np.int64)


@dataclass
class RecordTable:
    """Host arrays of a replay buffer in FIFO slot order (slot 0 oldest)."""
    length: np.ndarray      # int64 [n]
    arena_off: np.ndarray   # int64 [n]
    reward: np.ndarray      # float32 [n], 0/1
    version: np.ndarray     # int32 [n]
    group_off: np.ndarray   # int32 [n_groups + 1]
    cur_version: int


def record_table(wl, seed, n_records=None):
    """Record metadata: groups of G consecutive records share a prompt; each
    record has a length, a Bernoulli reward and a generating policy version
    (current version minus an age in U{0..4})."""
    rng = np.random.default_rng([seed, 1])
    n = wl.n_records if n_records is None else n_records
    ln = lengths(wl, n, rng)
    off = np.zeros(n, dtype=np.int64)
    off[1:] = np.cumsum(ln)[:-1]
    reward = (rng.random(n) < wl.reward_p).astype(np.float32)
    cur = 10
    age = rng.integers(0, 5, n)
    version = (cur - age).astype(np.int32)
    n_groups = (n + wl.group - 1) // wl.group
    group_off = np.minimum(np.arange(n_groups + 1) * wl.group, n).astype(np.int32)
    return RecordTable(ln, off, reward, version, group_off, cur)


def arena_tokens(total, V, seed, device="cpu"):
    """Token ids of every stored rollout, uniform over the vocabulary."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 7919 + 3)
    return torch.randint(0, V, (int(total),), generator=g, dtype=torch.int32, device=device)


def normal(shape, sd, seed, device="cpu", dtype=torch.float32):
    """N(0, sd^2) draws (e.g. staleness noise of stored log-probs)."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 104729 + 11)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    return (x * sd).to(dtype)


def head(T, d, V, seed, w_sd=0.02, device="cpu"):
    """hidden bf16 [T, d] ~ N(0, 1), W bf16 [V, d] ~ N(0, w_sd^2), tokens int32 [T]."""
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 1000003 + 17)
    hidden = torch.randn((T, d), generator=g, device=device).to(torch.bfloat16)
    W = (torch.randn((V, d), generator=g, device=device) * w_sd).to(torch.bfloat16)
    tokens = torch.randint(0, V, (T,), generator=g, dtype=torch.int32, device=device)
    return hidden, W, tokens


def uniform(shape, lo, hi, seed, device="cpu"):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) * 15485863 + 5)
    return lo + (hi - lo) * torch.rand(shape, generator=g, device=device)
