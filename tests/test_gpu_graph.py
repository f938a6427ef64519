"""The replay step as a HIP graph: sample + gather, log-prob forward, loss and
backward captured once (the library allocates nothing and never
synchronises, so every call is capturable), then replayed several times with
eager work and synchronisations in between; every replay must reproduce the
eager step bit for bit (all kernels are deterministic)."""

import numpy as np
import pytest
import torch

from paper_2604_08706_amd import workloads as wlm

from gpu_util import DeviceRing, require_gpu

pytestmark = pytest.mark.gpu


def _setup(rbp, T=2048, d=128, V=5000, n_draw=64):
    rng = np.random.default_rng(21)
    n = 300
    length = rng.integers(1, 65, n)
    off = np.concatenate([[0], np.cumsum(length)[:-1]])
    total = int(length.sum())
    ring = DeviceRing(rbp, length, off, (rng.random(n) < 0.4).astype(np.float32),
                      rng.standard_normal(n).astype(np.float32), rng.integers(0, 5, n),
                      rng.integers(0, V, total).astype(np.int32),
                      (rng.standard_normal(total) - 8.0).astype(np.float32), head=77,
                      capacity=400)
    cfg = rbp.make_sample_cfg(rbp.RB_UNIFORM, rbp.RB_LAYOUT_PACKED, 5, 3, n_draw, cur_version=6,
                              max_tokens=T)
    bufs = {
        "out": rbp.alloc_batch(cfg),
        "ws_s": rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, ring.capacity),
        "ws_f": rbp.workspace(rbp.RBP_OP_LOGPROB_FWD, T, d, V),
        "ws_l": rbp.workspace(rbp.RBP_OP_LOSS, T),
        "ws_b": rbp.workspace(rbp.RBP_OP_LOGPROB_BWD, T, d, V),
        "logp": torch.empty(T, device="cuda"), "lse": torch.empty(T, device="cuda"),
        "loss": torch.zeros(1, device="cuda"), "stats": torch.zeros(4, device="cuda"),
        "dlogp": torch.empty(T, device="cuda"),
        "dh": torch.empty((T, d), device="cuda"), "dW": torch.empty((V, d), device="cuda"),
    }
    hidden, W, _ = wlm.head(T, d, V, seed=22, device="cuda")
    return ring, cfg, bufs, hidden, W


def _step(rbp, ring, cfg, b, hidden, W):
    out = b["out"]
    rbp.rb_sample_gather(ring.rec, cfg, out, b["ws_s"])
    rbp.policy_logprob_fwd(hidden, W, out["tokens"], out["seq_of_token"], b["logp"], b["lse"],
                           b["ws_f"])
    b["loss"].zero_()  # a fill kernel, not a memset node
    b["stats"].zero_()
    rbp.policy_loss_fwd_bwd(b["logp"], out["old_logp"], out["seq_of_token"], out["adv"],
                            out["len"], cfg.n_draw, b["loss"], b["dlogp"], b["stats"], b["ws_l"])
    rbp.policy_logprob_bwd(hidden, W, out["tokens"], out["seq_of_token"], b["lse"], b["dlogp"],
                           b["dh"], b["dW"], b["ws_b"])


def _snapshot(b):
    keys = ("logp", "lse", "loss", "stats", "dlogp", "dh", "dW")
    snap = {k: b[k].clone() for k in keys}
    for k in ("idx", "tokens", "old_logp", "seq_of_token", "cu_seqlens", "n_tokens"):
        snap[k] = b["out"][k].clone()
    return snap


def test_replay_step_as_a_graph():
    rbp = require_gpu()
    ring, cfg, b, hidden, W = _setup(rbp)
    print("[graph] eager step", flush=True)
    _step(rbp, ring, cfg, b, hidden, W)
    torch.cuda.synchronize()
    want = _snapshot(b)
    assert int(want["n_tokens"].item()) > 1000
    # warm-up on a side stream, as torch's capture expects, then capture
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        _step(rbp, ring, cfg, b, hidden, W)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    print("[graph] capture", flush=True)
    with torch.cuda.graph(g):
        _step(rbp, ring, cfg, b, hidden, W)
    torch.cuda.synchronize()
    for r in range(3):
        # scribble over every output eagerly, then replay
        for k in ("logp", "lse", "dlogp", "dh", "dW"):
            b[k].fill_(float("nan"))
        b["out"]["tokens"].fill_(-7)
        b["loss"].fill_(123.0)
        torch.cuda.synchronize()
        print(f"[graph] replay {r}", flush=True)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(b)
        for k, v in want.items():
            assert torch.equal(got[k], v), (r, k)


def _fused_step(rbp, ring, cfg, b, hidden, W, ex):
    out = b["out"]
    rbp.rb_sample_gather(ring.rec, cfg, out, b["ws_s"])
    b["loss"].zero_()
    b["stats"].zero_()
    rbp.policy_fused_fwd_bwd(hidden, W, out["tokens"], out["seq_of_token"], out["old_logp"],
                             out["adv"], out["len"], cfg.n_draw, b["logp"], b["lse"], b["ent"],
                             b["loss"], b["dlogp"], b["stats"], b["dh"], b["dW"], b["ws_u"],
                             exec=ex)


@pytest.mark.parametrize("T,d,V,n_draw", [(2048, 128, 5000, 64), (9316, 1024, 3001, 400)])
def test_fused_step_as_a_graph(T, d, V, n_draw):
    """The single pass captured in a graph (its listed-token count is cleared
    by a kernel, not a memset node) replays bit for bit like the eager call;
    the second shape's dhidden (148 tiles) runs its round in K pieces."""
    rbp = require_gpu()
    ring, cfg, b, hidden, W = _setup(rbp, T, d, V, n_draw)
    T, d = hidden.shape
    V = W.shape[0]
    b["ent"] = torch.empty(T, device="cuda")
    b["ws_u"] = rbp.workspace(rbp.RBP_OP_FUSED, T, d, V)
    ex = None
    print("[graph] fused eager step", flush=True)
    _fused_step(rbp, ring, cfg, b, hidden, W, ex)
    torch.cuda.synchronize()
    want = _snapshot(b)
    want["ent"] = b["ent"].clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        _fused_step(rbp, ring, cfg, b, hidden, W, ex)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    print("[graph] fused capture", flush=True)
    with torch.cuda.graph(g):
        _fused_step(rbp, ring, cfg, b, hidden, W, ex)
    torch.cuda.synchronize()
    for r in range(3):
        for k in ("logp", "lse", "dlogp", "dh", "dW", "ent"):
            b[k].fill_(float("nan"))
        b["out"]["tokens"].fill_(-7)
        b["loss"].fill_(123.0)
        torch.cuda.synchronize()
        print(f"[graph] fused replay {r}", flush=True)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(b)
        got["ent"] = b["ent"].clone()
        for k, v in want.items():
            assert torch.equal(got[k], v), (r, k)
