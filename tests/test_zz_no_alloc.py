"""rb_sample_gather_noalloc (the library's static per-GPU scratch as the
workspace) against rb_sample_gather with a caller workspace: every output
bit for bit, on calls in a row whose inputs shrink, so that the second call
finds the first one's leftovers in the scratch; and the host-side rejection
of record tables too large for the scratch."""

import numpy as np
import pytest
import torch

from gpu_util import DeviceRing, require_gpu

pytestmark = pytest.mark.gpu

KEYS = ("idx", "adv", "len", "age", "cu_seqlens", "tokens", "old_logp", "seq_of_token",
        "n_tokens")


def _ring(rbp, n, cap, head, seed):
    rng = np.random.default_rng(seed)
    length = rng.integers(1, 300, n)
    off = np.concatenate([[0], np.cumsum(length)[:-1]])
    total = int(length.sum())
    return DeviceRing(rbp, length, off, (rng.random(n) < 0.35).astype(np.float32),
                      rng.standard_normal(n).astype(np.float32), rng.integers(0, 5, n),
                      rng.integers(0, 152064, total).astype(np.int32),
                      rng.standard_normal(total).astype(np.float32), head=head, capacity=cap)


def _compare(rbp, rec, cfg):
    ref = rbp.alloc_batch(cfg)
    got = rbp.alloc_batch(cfg)
    for v in got.values():  # the no-alloc call must write everything it returns
        v.fill_(-3) if v.dtype != torch.float32 else v.fill_(float("nan"))
    rbp.rb_sample_gather(rec, cfg, ref, rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, rec.capacity))
    rbp.rb_sample_gather_noalloc(rec, cfg, got)
    torch.cuda.synchronize()
    n_tok = int(ref["n_tokens"].item())
    assert int(got["n_tokens"].item()) == n_tok
    for k in KEYS:
        a, b = ref[k], got[k]  # padding included: both layouts define every position
        assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                           b.view(torch.int32) if b.dtype == torch.float32 else b), k


def test_noalloc_matches_workspace_call_on_shrinking_inputs():
    rbp = require_gpu()
    cases = [
        # (records, capacity, head, mode, layout, n_draw, extra cfg)
        (300_000, 320_000, 319_000, rbp.RB_NO_REPLACE, rbp.RB_LAYOUT_PADDED, 256,
         {"l_max": 512}),
        (1_000, 1_000, 17, rbp.RB_POS_MIX, rbp.RB_LAYOUT_PACKED, 20,
         {"max_tokens": 3000, "p_pos_q32": int(0.7 * 2 ** 32)}),
        (50_000, 60_000, 59_990, rbp.RB_UNIFORM, rbp.RB_LAYOUT_PACKED, 2000,
         {"max_tokens": 16384, "token_begin": 1234}),
        (64, 64, 0, rbp.RB_POS_RETAIN, rbp.RB_LAYOUT_PADDED, 8,
         {"l_max": 300, "n_fresh": 32, "n_pos_keep": 16}),
    ]
    for i, (n, cap, head, mode, layout, n_draw, extra) in enumerate(cases):
        print(f"[noalloc] call {i}: n={n} cap={cap} mode={mode} layout={layout} "
              f"n_draw={n_draw}", flush=True)
        ring = _ring(rbp, n, cap, head, 100 + i)
        cfg = rbp.make_sample_cfg(mode, layout, 9, 4 + i, n_draw, cur_version=7, **extra)
        _compare(rbp, ring.rec, cfg)
        del ring
    torch.cuda.empty_cache()


def test_noalloc_rejects_tables_beyond_its_scratch():
    rbp = require_gpu()
    ring = _ring(rbp, 10, 10, 0, 5)
    cfg = rbp.make_sample_cfg(rbp.RB_UNIFORM, rbp.RB_LAYOUT_PACKED, 1, 0, 4, max_tokens=100)
    out = rbp.alloc_batch(cfg)
    cap = 2_000_000
    z = lambda dt: torch.zeros(cap, dtype=dt, device="cuda")  # noqa: E731
    big = rbp.make_records(10, cap, 0, z(torch.int64), z(torch.int32) + 1, z(torch.float32),
                           z(torch.float32), z(torch.int32), ring.t_tok, ring.t_old)
    assert rbp.rbp_workspace_bytes(rbp.RBP_OP_SAMPLE_GATHER, 2_000_000) > 32 << 20
    with pytest.raises(rbp.RbpError) as e:
        rbp.rb_sample_gather_noalloc(big, cfg, out)  # refused on the host, nothing enqueued
    assert e.value.status == rbp.RBP_EWORKSPACE
    assert "static scratch" in str(e.value)
    # the largest table it takes
    ok = rbp.rbp_workspace_bytes(rbp.RBP_OP_SAMPLE_GATHER, 1_500_000) <= 32 << 20
    assert ok


def _largest_capacity(rbp, limit=32 << 20):
    lo, hi = 1, 1 << 24
    while lo < hi:  # largest capacity whose workspace fits the scratch
        mid = (lo + hi + 1) // 2
        if rbp.rbp_workspace_bytes(rbp.RBP_OP_SAMPLE_GATHER, mid) <= limit:
            lo = mid
        else:
            hi = mid - 1
    return lo


def test_noalloc_at_the_largest_table_its_scratch_holds():
    """The largest record table the 32 MiB scratch holds (every slot live, the
    ring's head inside it) matches the workspace call bit for bit, without
    and with replacement; one slot more is refused on the host."""
    rbp = require_gpu()
    cap = _largest_capacity(rbp)
    print(f"[noalloc] largest capacity {cap}", flush=True)
    assert 1_500_000 < cap < 1_700_000
    rng = np.random.default_rng(77)
    length = rng.integers(1, 5, cap)
    off = np.concatenate([[0], np.cumsum(length)[:-1]])
    total = int(length.sum())
    ring = DeviceRing(rbp, length, off, (rng.random(cap) < 0.4).astype(np.float32),
                      rng.standard_normal(cap).astype(np.float32), rng.integers(0, 5, cap),
                      rng.integers(0, 152064, total).astype(np.int32),
                      rng.standard_normal(total).astype(np.float32), head=cap // 3,
                      capacity=cap)
    for mode, layout, n_draw, extra in (
            (rbp.RB_NO_REPLACE, rbp.RB_LAYOUT_PADDED, 512, {"l_max": 8}),
            (rbp.RB_UNIFORM, rbp.RB_LAYOUT_PACKED, 4096, {"max_tokens": 8192})):
        cfg = rbp.make_sample_cfg(mode, layout, 3, 11, n_draw, cur_version=7, **extra)
        _compare(rbp, ring.rec, cfg)
    big = rbp.make_records(cap, cap + 1, 0, torch.cat([ring.t_off, ring.t_off[:1]]),
                           torch.cat([ring.t_len, ring.t_len[:1]]),
                           torch.cat([ring.t_rew, ring.t_rew[:1]]),
                           torch.cat([ring.t_adv, ring.t_adv[:1]]),
                           torch.cat([ring.t_ver, ring.t_ver[:1]]), ring.t_tok, ring.t_old)
    cfg = rbp.make_sample_cfg(rbp.RB_UNIFORM, rbp.RB_LAYOUT_PACKED, 1, 0, 4, max_tokens=100)
    with pytest.raises(rbp.RbpError) as e:
        rbp.rb_sample_gather_noalloc(big, cfg, rbp.alloc_batch(cfg))
    assert e.value.status == rbp.RBP_EWORKSPACE
    del ring, big
    torch.cuda.empty_cache()
