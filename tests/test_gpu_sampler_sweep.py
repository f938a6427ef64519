"""Seeded sweep of rb_sample_gather against the oracle, bit for bit: random
table sizes, ring capacities and heads, sampling rules and their parameters,
draw counts on both sides of the single-block limit (1024), and packed
windows or padded rows of random extent."""

import numpy as np
import pytest

from oracle import buffer as ob
from oracle import philox
from paper_2604_08706_amd import workloads as wlm

from gpu_util import DeviceRing, require_gpu
import test_gpu_sampler as smp

pytestmark = pytest.mark.gpu


def _cases(n=30, seed=77):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        n_rec = int(rng.integers(1, 5001))
        cap = n_rec + int(rng.integers(0, 300))
        head = int(rng.integers(0, cap))
        mode = ["uniform", "pos_mix", "pos_retain"][i % 3]
        layout = ["packed", "padded"][(i // 3) % 2]
        n_draw = int(rng.integers(1, 3001))
        out.append((i, n_rec, cap, head, mode, layout, n_draw))
    return out


@pytest.mark.parametrize("i,n_rec,cap,head,mode,layout,n_draw", _cases())
def test_sampler_sweep(i, n_rec, cap, head, mode, layout, n_draw):
    rbp = require_gpu()
    rng = np.random.default_rng([i, 5])
    wl = wlm.WORKLOADS["head05b"] if i % 2 else wlm.WORKLOADS["tiny"]
    tab, tok, old, adv = smp._host_table(wl, 100 + i, n_rec)
    ring = DeviceRing(rbp, tab.length, tab.arena_off, tab.reward, adv, tab.version, tok, old,
                      head=head, capacity=cap)
    p = float(rng.random())
    n_fresh, n_pos_keep = ob.retain_split(n_rec, float(rng.random()))
    kw = dict(p_q32=philox.p_to_q32(p) if mode == "pos_mix" else 0,
              n_fresh=n_fresh if mode == "pos_retain" else 0,
              n_pos_keep=n_pos_keep if mode == "pos_retain" else 0)
    seed, step = int(rng.integers(0, 2**31)), int(rng.integers(0, 10**6))
    if layout == "packed":
        lk = dict(max_tokens=int(rng.integers(1, 20001)),
                  token_begin=int(rng.integers(0, 20001)))
    else:
        lk = dict(l_max=int(rng.integers(1, 1500)))
    got = smp._run(rbp, ring, mode, layout, seed, step, n_draw, **kw, **lk)
    want = smp._oracle(tab, tok, old, adv, mode, layout, seed, step, n_draw, **kw, **lk)
    smp._compare(got, want)
