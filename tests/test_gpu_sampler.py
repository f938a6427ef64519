"""GPU parity of rb_sample_gather against the oracle: bit-exact indices and
gathered bytes, every mode and layout, ring heads, micro-batch windows, and the
full-size record tables of the benchmark workloads."""

import numpy as np
import pytest
import torch

from oracle import buffer as ob
from oracle import philox
from paper_2604_08706_amd import workloads as wlm

from gpu_util import DeviceRing, require_gpu, to_np

pytestmark = pytest.mark.gpu

MODES = {"uniform": ob.RB_UNIFORM, "pos_mix": ob.RB_POS_MIX, "pos_retain": ob.RB_POS_RETAIN}


def _host_table(wl, seed, n_records=None):
    tab = wlm.record_table(wl, seed, n_records)
    total = int(tab.length.sum())
    tok = wlm.arena_tokens(total, wl.V, seed).numpy()
    old = wlm.normal(total, 1.0, seed + 1).numpy()
    adv = wlm.normal(len(tab.length), 1.0, seed + 2).numpy()
    return tab, tok, old, adv


def _run(rbp, ring, mode, layout, seed, step, n_draw, p_q32=0, n_fresh=0, n_pos_keep=0,
         cur_version=10, max_tokens=0, token_begin=0, l_max=0):
    lay = rbp.RB_LAYOUT_PACKED if layout == "packed" else rbp.RB_LAYOUT_PADDED
    cfg = rbp.make_sample_cfg(MODES[mode], lay, seed, step, n_draw, p_q32, n_fresh,
                              n_pos_keep, cur_version, max_tokens, token_begin, l_max)
    out = rbp.alloc_batch(cfg)
    ws = rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, ring.capacity)
    print(f"[sampler] mode={mode} layout={layout} seed={seed} step={step} n_draw={n_draw}",
          flush=True)
    rbp.rb_sample_gather(ring.rec, cfg, out, ws)
    torch.cuda.synchronize()
    return {k: to_np(v) for k, v in out.items()}


def _oracle(tab, tok, old, adv, mode, layout, seed, step, n_draw, p_q32=0, n_fresh=0,
            n_pos_keep=0, cur_version=10, max_tokens=0, token_begin=0, l_max=0):
    idx = ob.sample_indices(tab.reward, MODES[mode], seed, step, n_draw, p_q32, n_fresh,
                            n_pos_keep)
    lay = ob.LAYOUT_PACKED if layout == "packed" else ob.LAYOUT_PADDED
    return ob.gather(idx, tab.arena_off, tab.length, adv, tab.version, tok, old, cur_version,
                     lay, max_tokens, token_begin, l_max)


def _compare(got, want):
    for k in ("idx", "len", "age", "cu_seqlens"):
        assert np.array_equal(got[k], want[k]), k
    assert np.array_equal(got["adv"].view(np.int32), want["adv"].view(np.int32))
    assert got["n_tokens"][0] == want["n_tokens"]
    for k in ("tokens", "seq_of_token"):
        assert np.array_equal(got[k].reshape(-1), want[k].reshape(-1)), k
    assert np.array_equal(got["old_logp"].reshape(-1).view(np.int32),
                          want["old_logp"].reshape(-1).view(np.int32))


@pytest.mark.parametrize("mode,p,delta", [
    ("uniform", 0, 0), ("pos_mix", 0.0, 0), ("pos_mix", 0.5, 0), ("pos_mix", 1.0, 0),
    ("pos_retain", 0, 0.0), ("pos_retain", 0, 0.5), ("pos_retain", 0, 0.25),
])
@pytest.mark.parametrize("layout", ["padded", "packed"])
def test_tiny_all_modes_bit_exact(mode, p, delta, layout):
    rbp = require_gpu()
    wl = wlm.WORKLOADS["tiny"]
    tab, tok, old, adv = _host_table(wl, 0)
    ring = DeviceRing(rbp, tab.length, tab.arena_off, tab.reward, adv, tab.version, tok, old,
                      head=37, capacity=100)
    n_fresh, n_pos_keep = ob.retain_split(48, delta)
    kw = dict(p_q32=philox.p_to_q32(p), n_fresh=n_fresh, n_pos_keep=n_pos_keep)
    for step in (0, 3):
        if layout == "padded":
            lk = dict(l_max=32)
            got = _run(rbp, ring, mode, layout, 0, step, 8, **kw, **lk)
            want = _oracle(tab, tok, old, adv, mode, layout, 0, step, 8, **kw, **lk)
            _compare(got, want)
        else:
            for tb in (0, 70, 10_000):
                lk = dict(max_tokens=100, token_begin=tb)
                got = _run(rbp, ring, mode, layout, 0, step, 8, **kw, **lk)
                want = _oracle(tab, tok, old, adv, mode, layout, 0, step, 8, **kw, **lk)
                _compare(got, want)


def test_paper_worked_example_on_gpu():
    # App. D.4 example (10 rollouts, N = 8, delta = 0.5): every draw lands in
    # the printed buffer and all 8 of its members are drawn
    rbp = require_gpu()
    correct = np.array([0, 1, 1, 0, 1, 1, 0, 1, 0, 0], dtype=np.float32)
    n = len(correct)
    length = np.full(n, 3)
    off = np.arange(n) * 3
    tok = np.arange(3 * n, dtype=np.int32)
    old = np.zeros(3 * n, dtype=np.float32)
    ring = DeviceRing(rbp, length, off, correct, np.zeros(n), np.zeros(n), tok, old, head=5)
    got = _run(rbp, ring, "pos_retain", "padded", 9, 0, 4000, n_fresh=4, n_pos_keep=4, l_max=3)
    assert set(got["idx"].tolist()) == {1, 2, 4, 5, 6, 7, 8, 9}


def test_head05b_uniform_packed_windows():
    rbp = require_gpu()
    wl = wlm.WORKLOADS["head05b"]
    tab, tok, old, adv = _host_table(wl, 1)
    ring = DeviceRing(rbp, tab.length, tab.arena_off, tab.reward, adv, tab.version, tok, old,
                      head=1234, capacity=5000)
    for step, tb in [(0, 0), (0, 16384), (5, 0)]:
        kw = dict(max_tokens=wl.max_tokens, token_begin=tb)
        got = _run(rbp, ring, "uniform", "packed", 1, step, wl.n_draw, **kw)
        want = _oracle(tab, tok, old, adv, "uniform", "packed", 1, step, wl.n_draw, **kw)
        _compare(got, want)


def test_head15b_positive_mixture():
    rbp = require_gpu()
    wl = wlm.WORKLOADS["head15b"]
    tab, tok, old, adv = _host_table(wl, 2)
    ring = DeviceRing(rbp, tab.length, tab.arena_off, tab.reward, adv, tab.version, tok, old,
                      head=32767, capacity=32768)
    p = philox.p_to_q32(wl.p_pos)
    got = _run(rbp, ring, "pos_mix", "packed", 2, 7, wl.n_draw, p_q32=p, max_tokens=16384,
               token_begin=16384 * 3)
    want = _oracle(tab, tok, old, adv, "pos_mix", "packed", 2, 7, wl.n_draw, p_q32=p,
                   max_tokens=16384, token_begin=16384 * 3)
    _compare(got, want)
    frac = tab.reward[got["idx"]].mean()
    assert frac > 0.6  # p + (1 - p) f_pos ~ 0.79


def test_head7b_micro_batch_is_full():
    rbp = require_gpu()
    wl = wlm.WORKLOADS["head7b"]
    tab, tok, old, adv = _host_table(wl, 0)
    ring = DeviceRing(rbp, tab.length, tab.arena_off, tab.reward, adv, tab.version, tok, old)
    kw = dict(max_tokens=16384, token_begin=0)
    got = _run(rbp, ring, "uniform", "packed", 0, 0, wl.n_draw, **kw)
    want = _oracle(tab, tok, old, adv, "uniform", "packed", 0, 0, wl.n_draw, **kw)
    _compare(got, want)
    assert got["n_tokens"][0] == 16384


def test_stress_million_records_padded():
    """10^6 records, ~1.8e9 arena tokens in HBM, 256 mixed draws, padded to
    8192; then 256 draws without replacement, as the benchmark times them."""
    rbp = require_gpu()
    wl = wlm.WORKLOADS["stress"]
    tab = wlm.record_table(wl, 3)
    total = int(tab.length.sum())
    tok_d = wlm.arena_tokens(total, wl.V, 3, device="cuda")
    old_d = wlm.normal(total, 1.0, 4, device="cuda")
    adv = wlm.normal(len(tab.length), 1.0, 5).numpy()
    ring = DeviceRing(rbp, tab.length, tab.arena_off, tab.reward, adv, tab.version, tok_d,
                      old_d, head=999_000, capacity=1_048_576)
    p = philox.p_to_q32(wl.p_pos)
    got = _run(rbp, ring, "pos_mix", "padded", 3, 11, wl.n_draw, p_q32=p, l_max=wl.l_max)
    idx = ob.sample_indices(tab.reward, ob.RB_POS_MIX, 3, 11, wl.n_draw, p)
    assert np.array_equal(got["idx"], np.array(idx, dtype=np.int32))
    _compare(got, _compact_gather(idx, tab, tok_d, old_d, adv, wl.l_max))
    # the benchmark's draw without replacement on the same buffer (seed 3,
    # step 0, padded): a radix select over all 10^6 slot keys
    cfg = rbp.make_sample_cfg(rbp.RB_NO_REPLACE, rbp.RB_LAYOUT_PADDED, 3, 0, wl.n_draw,
                              cur_version=tab.cur_version, l_max=wl.l_max)
    out = rbp.alloc_batch(cfg)
    print("[sampler] stress no_replace n_live=10^6 n_draw=256", flush=True)
    rbp.rb_sample_gather(ring.rec, cfg, out, rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER,
                                                           ring.capacity))
    torch.cuda.synchronize()
    got = {k: to_np(v) for k, v in out.items()}
    idx = ob.sample_without_replacement(3, 0, len(tab.length), wl.n_draw)
    assert np.array_equal(got["idx"], np.array(idx, dtype=np.int32))
    _compare(got, _compact_gather(idx, tab, tok_d, old_d, adv, wl.l_max))
    del tok_d, old_d, out
    torch.cuda.empty_cache()


def _compact_gather(idx, tab, tok_d, old_d, adv, l_max):
    """The oracle's padded gather over a compact arena holding only the drawn
    records (the full arena is too large to copy to the host)."""
    c_off, chunks_t, chunks_o, at = {}, [], [], 0
    for s in sorted(set(idx)):
        a, n = int(tab.arena_off[s]), int(min(tab.length[s], l_max))
        chunks_t.append(to_np(tok_d[a:a + n]))
        chunks_o.append(to_np(old_d[a:a + n]))
        c_off[s] = at
        at += n
    off2 = np.zeros(len(tab.length), dtype=np.int64)
    for s, o in c_off.items():
        off2[s] = o
    return ob.gather(idx, off2, tab.length, adv, tab.version, np.concatenate(chunks_t),
                     np.concatenate(chunks_o), tab.cur_version, ob.LAYOUT_PADDED, l_max=l_max)


def test_same_seed_step_reproduces_and_rejects_bad_args():
    rbp = require_gpu()
    wl = wlm.WORKLOADS["tiny"]
    tab, tok, old, adv = _host_table(wl, 0)
    ring = DeviceRing(rbp, tab.length, tab.arena_off, tab.reward, adv, tab.version, tok, old)
    a = _run(rbp, ring, "uniform", "padded", 4, 2, 8, l_max=32)
    b = _run(rbp, ring, "uniform", "padded", 4, 2, 8, l_max=32)
    for k in a:
        assert np.array_equal(a[k], b[k])
    cfg = rbp.make_sample_cfg(7, rbp.RB_LAYOUT_PADDED, 0, 0, 8, l_max=32)
    with pytest.raises(rbp.RbpError) as e:
        rbp.rb_sample_gather(ring.rec, cfg, rbp.alloc_batch(
            rbp.make_sample_cfg(0, 1, 0, 0, 8, l_max=32)),
            rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, ring.capacity))
    assert e.value.status == rbp.RBP_EINVAL
    cfg = rbp.make_sample_cfg(0, rbp.RB_LAYOUT_PADDED, 0, 0, 8, l_max=32)
    small = torch.empty(8, dtype=torch.uint8, device="cuda")
    with pytest.raises(rbp.RbpError) as e:
        rbp.rb_sample_gather(ring.rec, cfg, rbp.alloc_batch(cfg), small)
    assert e.value.status == rbp.RBP_EWORKSPACE


def _small_records(n, seed):
    """n records of 1..8 tokens, about 30 % positive, versions 0..9."""
    rng = np.random.default_rng(seed)
    length = rng.integers(1, 9, n)
    off = np.concatenate([[0], np.cumsum(length)[:-1]])
    total = int(length.sum())
    return dict(length=length, arena_off=off, reward=(rng.random(n) < 0.3).astype(np.float32),
                adv=rng.standard_normal(n).astype(np.float32), version=rng.integers(0, 10, n),
                tok=rng.integers(0, 1000, total).astype(np.int32),
                old=rng.standard_normal(total).astype(np.float32))


@pytest.mark.parametrize("mode,layout", [
    ("uniform", "packed"), ("pos_mix", "padded"), ("pos_retain", "packed")])
def test_many_draws_carry_the_length_prefix_across_rounds(mode, layout):
    # 20000 draws: the per-draw pass runs several rounds of 4096 draws and
    # carries the packed offsets from one round to the next
    rbp = require_gpu()
    r = _small_records(3000, 8)
    ring = DeviceRing(rbp, r["length"], r["arena_off"], r["reward"], r["adv"], r["version"],
                      r["tok"], r["old"], head=2999, capacity=3500)
    n_fresh, n_pos_keep = ob.retain_split(3000, 0.25)
    kw = dict(p_q32=philox.p_to_q32(0.5), n_fresh=n_fresh, n_pos_keep=n_pos_keep)
    lk = dict(max_tokens=200_000) if layout == "packed" else dict(l_max=8)
    got = _run(rbp, ring, mode, layout, 6, 2, 20_000, **kw, **lk)
    idx = ob.sample_indices(r["reward"], MODES[mode], 6, 2, 20_000, **kw)
    lay = ob.LAYOUT_PACKED if layout == "packed" else ob.LAYOUT_PADDED
    want = ob.gather(idx, r["arena_off"], r["length"], r["adv"], r["version"], r["tok"],
                     r["old"], 10, lay, **lk)
    _compare(got, want)


def test_without_replacement_many_draws_match_oracle():
    # 9000 of 10000 records: the select's bucket holds most keys and the
    # per-draw pass runs three rounds
    rbp = require_gpu()
    r = _small_records(10_000, 9)
    ring = DeviceRing(rbp, r["length"], r["arena_off"], r["reward"], r["adv"], r["version"],
                      r["tok"], r["old"], head=77, capacity=10_000)
    cfg = rbp.make_sample_cfg(rbp.RB_NO_REPLACE, rbp.RB_LAYOUT_PACKED, 5, 1, 9000,
                              cur_version=10, max_tokens=80_000)
    out = rbp.alloc_batch(cfg)
    print("[sampler] no_replace n_live=10000 n_draw=9000", flush=True)
    rbp.rb_sample_gather(ring.rec, cfg, out, rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, 10_000))
    torch.cuda.synchronize()
    got = {k: to_np(v) for k, v in out.items()}
    idx = ob.sample_without_replacement(5, 1, 10_000, 9000)
    want = ob.gather(idx, r["arena_off"], r["length"], r["adv"], r["version"], r["tok"],
                     r["old"], 10, ob.LAYOUT_PACKED, max_tokens=80_000)
    _compare(got, want)


def test_maximum_draw_count_packed():
    # n_draw = 2^20, the largest batch the call accepts: 4096 blocks of draws
    # and a scan over all their sums; the window stops inside the stream
    rbp = require_gpu()
    r = _small_records(5000, 10)
    ring = DeviceRing(rbp, r["length"], r["arena_off"], r["reward"], r["adv"], r["version"],
                      r["tok"], r["old"], head=4321, capacity=6000)
    n = 1 << 20
    lk = dict(max_tokens=3_000_000, token_begin=1_000_000)
    got = _run(rbp, ring, "uniform", "packed", 12, 3, n, **lk)
    idx = ob.sample_indices(r["reward"], ob.RB_UNIFORM, 12, 3, n)
    want = ob.gather(idx, r["arena_off"], r["length"], r["adv"], r["version"], r["tok"],
                     r["old"], 10, ob.LAYOUT_PACKED, **lk)
    _compare(got, want)


@pytest.mark.parametrize("n_fresh,n_pos_keep", [(0, 0), (0, 5)])
def test_pos_retain_empty_set_draws_slot_zero(n_fresh, n_pos_keep):
    """Positive-bias retention with an empty retained set (no fresh slots
    and no positive record to keep): the documented fallback draws logical
    slot 0 every time, and the batch is the gather of those draws."""
    rbp = require_gpu()
    wl = wlm.WORKLOADS["tiny"]
    tab, tok, old, adv = _host_table(wl, 3)
    reward = np.zeros_like(tab.reward)  # no positives
    ring = DeviceRing(rbp, tab.length, tab.arena_off, reward, adv, tab.version, tok, old,
                      head=11, capacity=80)
    kw = dict(n_fresh=n_fresh, n_pos_keep=n_pos_keep, l_max=40)
    got = _run(rbp, ring, "pos_retain", "padded", 4, 2, 16, **kw)
    assert np.all(got["idx"] == 0)
    want = ob.gather([0] * 16, tab.arena_off, tab.length, adv, tab.version, tok, old, 10,
                     ob.LAYOUT_PADDED, 0, 0, 40)
    _compare(got, want)
