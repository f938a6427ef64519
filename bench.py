"""Replayed-token throughput of the replay hot path on one MI355X.

One step = the whole trainer-side path over one replay micro-batch:
  rb_group_advantage    (advantages of the buffer's groups, as at insert)
  rb_sample_gather      (uniform draws from a 1024-record FIFO buffer, packed
                         into a 16384-token micro-batch)
  policy_fused_fwd_bwd  (one pass: logits hidden [16384, 3584] x W [152064,
                         3584] in bf16 MFMA tiles with the log-sum-exp
                         partials and q = exp(z - R_t) kept per tile (R_t the
                         token's reference), the clipped GRPO loss with
                         token ratios and group advantages, and the backward
                         to dhidden and dW, dW accumulated as over
                         micro-batches; 6 d V flop per token)
`value` is this step's throughput.  Reported beside it: the four-call step
(policy_logprob_fwd + policy_loss_fwd_bwd + policy_logprob_bwd, whose
backward recomputes the logits: 8 d V flop per token), and both paths with a
workspace bounded to 4096-token chunks.  Inputs are synthetic (seeded),
shaped like Qwen2.5-7B's LM head and the paper's rollout length mix; hidden
states stand in for the model trunk's output.  All inputs are resident in HBM
before timing starts.

Prints one JSON line (metric: replayed tokens/s; also the fraction of the
MI355X dense bf16 MFMA peak, per-phase times from the call's own events, a
roofline record for the product that takes the most time per step, and the
CPU oracle timed on a bounded sample).
"""

import argparse
import json
import os
import sys
import time

import numpy as np

PEAK_BF16 = 2.5e15        # MI355X dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12         # MI355X HBM3E, B/s
ROOT = os.path.dirname(os.path.abspath(__file__))

# HBM traffic per step of each product of the single pass at the 16384-token
# micro-batch (d=3584, V=152064): FETCH_SIZE and WRITE_SIZE per dispatch from
# two rocprofv3 --pmc passes over this script, scaled by what the same
# counters read for a plain copy of known size (--copy-probe-mib), summed over
# a product's launches in one step.  Only valid for the sources the counters
# were read on (None until they are).
TRAFFIC_SOURCES = ("fused.hip", "logprob_bwd.hip", "logits_epilogue.h", "gemm_core.h",
                   "gemm_dma.h", "advantage_loss.hip")
# FETCH_SIZE x 2.0 + WRITE_SIZE x 1.0 (a 1 GiB copy reads 524300 KiB of
# FETCH_SIZE and 1048576 KiB of WRITE_SIZE), per step:
#   logits  = target_ref_kernel + logits_store_kernel
#   dW      = dweight_kernel (main launch + last-round launch) + part_add_kernel
#   dhidden = dhidden_kernel (main launch + last-round launch) + part_add_dh_kernel
TRAFFIC = {
    "sources_sha256": "2825da243df2c1621cbac27110d208ee401acf8a4a769cfa1f4deb269e77941d",
    "bytes": {"logits": 34395098112, "dW": 42019896320, "dhidden": 40238567424},
}

# the three products of the single pass, by the phase that times them
PRODUCTS = {
    "logits": "logits_store_kernel (forward product; stores q = exp(z - R_t) as bf16)",
    "dW": "dweight_kernel (dW product)",
    "dhidden": "dhidden_kernel (dhidden product: main launch + last-round K halves)",
}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="head7b")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-tokens", type=int, default=3072,
                    help="tokens of the bounded sample the CPU oracle is timed on")
    ap.add_argument("--no-aux", action="store_true",
                    help="skip the HBM-rate measurement of sample+gather and loss on the "
                         "10^6-record stress buffer")
    ap.add_argument("--no-four-call", action="store_true",
                    help="skip the separately reported four-call leg")
    ap.add_argument("--no-bounded", action="store_true",
                    help="skip the bounded-workspace legs (both paths in chunks)")
    ap.add_argument("--bounded-tokens", type=int, default=4096,
                    help="token chunk the bounded-workspace legs size their workspace for")
    ap.add_argument("--blas-probe", action="store_true",
                    help="only time the vendor library's plain bf16 GEMM on the forward's "
                         "shape (W [V, d] x hidden^T [d, T], torch.mm) as a practical "
                         "ceiling, print one JSON line and exit")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a plain device-to-device copy of this many MiB three "
                         "times (calibrates the HBM byte counters) and exit")
    return ap.parse_args()


def copy_probe(mib):
    """A plain copy of known size, for scaling FETCH_SIZE / WRITE_SIZE."""
    import torch

    n = mib << 18  # float32 elements
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n * 4, "copy_probe_bytes_written": n * 4}))


def blas_probe(steps=10, warmup=3):
    """The three products of a replay step through torch.mm (hipBLASLt) at the
    7B head shape, bf16 in and out, every operand contiguous: the forward's
    Z^T = W H^T, dhidden = dZ W and dW = dZ^T H, each 2*T*d*V flop (no
    log-sum-exp, no dz epilogue, no accumulation).  A measurement of the
    vendor GEMM, not a product path."""
    import torch

    from paper_2604_08706_amd import workloads as wlm

    wl = wlm.WORKLOADS["head7b"]
    T = wl.max_tokens
    hidden, W, _ = wlm.head(T, wl.d, wl.V, 0, device="cuda")
    ht = hidden.t().contiguous()
    dz = (torch.randn((T, wl.V), device="cuda") * 1e-3).bfloat16()
    dzt = dz.t().contiguous()
    cases = [
        ("forward Z^T = W H^T: [V, d] x [d, T]", W, ht, (wl.V, T)),
        ("dhidden = dZ W: [T, V] x [V, d]", dz, W, (T, wl.d)),
        ("dW = dZ^T H: [V, T] x [T, d]", dzt, hidden, (wl.V, wl.d)),
    ]
    flop = 2.0 * T * wl.d * wl.V
    for name, a_, b_, shape in cases:
        out = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
        for _ in range(warmup):
            torch.mm(a_, b_, out=out)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            torch.mm(a_, b_, out=out)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / steps
        print(json.dumps({"probe": "torch.mm bf16 " + name, "T": T, "d": wl.d, "V": wl.V,
                          "ms": round(ms, 3), "TFLOP/s": round(flop / (ms / 1e3) / 1e12, 1),
                          "frac_peak": round(flop / (ms / 1e3) / PEAK_BF16, 4)}), flush=True)
        del out


def sources_sha256():
    import hashlib

    h = hashlib.sha256()
    for name in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, "paper_2604_08706_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_bytes(product):
    """HBM bytes per step of one product of the single pass, or None when
    not measured on the current kernel sources."""
    if TRAFFIC is None or TRAFFIC["sources_sha256"] != sources_sha256():
        return None
    return TRAFFIC["bytes"].get(product)


def setup(wl, seed=0):
    import torch

    import paper_2604_08706_amd as rbp
    from paper_2604_08706_amd import workloads as wlm

    dev = "cuda"
    T = wl.max_tokens
    tab = wlm.record_table(wl, seed)
    total = int(tab.length.sum())
    S = {}
    S["rewards"] = torch.from_numpy(tab.reward).to(dev)
    S["group_off"] = torch.from_numpy(tab.group_off).to(dev)
    S["adv_rec"] = torch.zeros(len(tab.length), dtype=torch.float32, device=dev)
    S["len_rec"] = torch.from_numpy(tab.length.astype(np.int32)).to(dev)
    S["off_rec"] = torch.from_numpy(tab.arena_off).to(dev)
    S["ver_rec"] = torch.from_numpy(tab.version).to(dev)
    S["arena_tok"] = wlm.arena_tokens(total, wl.V, seed, device=dev)
    S["arena_old"] = torch.zeros(total, dtype=torch.float32, device=dev)
    S["rec"] = rbp.make_records(len(tab.length), len(tab.length), 0, S["off_rec"], S["len_rec"],
                                S["rewards"], S["adv_rec"], S["ver_rec"], S["arena_tok"],
                                S["arena_old"])
    hidden, W, _ = wlm.head(T, wl.d, wl.V, seed, device=dev)
    S["hidden"], S["W"] = hidden, W
    S["dW"] = torch.zeros((wl.V, wl.d), dtype=torch.float32, device=dev)
    S["dh"] = torch.empty((T, wl.d), dtype=torch.float32, device=dev)
    S["logp"] = torch.empty(T, device=dev)
    S["lse"] = torch.empty(T, device=dev)
    S["dlogp"] = torch.empty(T, device=dev)
    S["loss"] = torch.zeros(1, device=dev)
    S["stats"] = torch.zeros(4, device=dev)
    S["ws_sample"] = rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, len(tab.length))
    S["ws_fwd"] = rbp.workspace(rbp.RBP_OP_LOGPROB_FWD, T, wl.d, wl.V)
    S["ws_loss"] = rbp.workspace(rbp.RBP_OP_LOSS, T)
    S["ws_bwd"] = rbp.workspace(rbp.RBP_OP_LOGPROB_BWD, T, wl.d, wl.V)
    S["T"] = T
    S["tab"] = tab
    return S


def cfg_for(rbp, wl, step, seed=0):
    return rbp.make_sample_cfg(rbp.RB_UNIFORM, rbp.RB_LAYOUT_PACKED, seed, step, wl.n_draw,
                               cur_version=10, max_tokens=wl.max_tokens, token_begin=0)


def align_old_logp(rbp, wl, S, steps, noise_sd, seed=0):
    """Untimed: store behaviour log-probs for the tokens each step will draw,
    as the current policy's log-probs plus staleness noise (a replayed,
    slightly stale rollout)."""
    import torch

    from paper_2604_08706_amd import workloads as wlm

    for k in steps:
        cfg = cfg_for(rbp, wl, k, seed)
        out = rbp.alloc_batch(cfg)
        rbp.rb_sample_gather(S["rec"], cfg, out, S["ws_sample"])
        rbp.policy_logprob_fwd(S["hidden"], S["W"], out["tokens"], out["seq_of_token"],
                               S["logp"], S["lse"], S["ws_fwd"])
        seq = out["seq_of_token"].long()
        ok = seq >= 0
        pos = torch.arange(S["T"], device="cuda")
        start = out["cu_seqlens"].long()[seq.clamp(min=0)]
        src = S["off_rec"][out["idx"].long()[seq.clamp(min=0)]] + (pos - start)
        noise = wlm.normal(S["T"], noise_sd, 1000 + k, device="cuda")
        S["arena_old"][src[ok]] = (S["logp"] + noise)[ok]
    torch.cuda.synchronize()


def run_step(rbp, wl, S, step, out, ev=None, ws_bwd=None):
    """The four-call step.  ev: 5 timing events (step start, after the
    sampler, after the forward, after the loss, after the backward)."""
    if ev is not None:
        ev[0].record()
    rbp.rb_group_advantage(S["rewards"], S["group_off"], S["adv_rec"])
    rbp.rb_sample_gather(S["rec"], cfg_for(rbp, wl, step), out, S["ws_sample"])
    if ev is not None:
        ev[1].record()
    rbp.policy_logprob_fwd(S["hidden"], S["W"], out["tokens"], out["seq_of_token"], S["logp"],
                           S["lse"], S["ws_fwd"])
    if ev is not None:
        ev[2].record()
    rbp.policy_loss_fwd_bwd(S["logp"], out["old_logp"], out["seq_of_token"], out["adv"],
                            out["len"], wl.n_draw, S["loss"], S["dlogp"], S["stats"],
                            S["ws_loss"])
    if ev is not None:
        ev[3].record()
    rbp.policy_logprob_bwd(S["hidden"], S["W"], out["tokens"], out["seq_of_token"], S["lse"],
                           S["dlogp"], S["dh"], S["dW"], S["ws_bwd"] if ws_bwd is None else ws_bwd,
                           accumulate_dW=True)
    if ev is not None:
        ev[4].record()


def aux_stress(iters=20):
    """HBM rate of the two memory-bound steps on the long-sequence stress
    buffer (10^6 records, ~1.8e9 stored tokens in HBM):
      sample+gather: 256 positive-mixture draws (p_pos = 0.5), padded to 8192;
      loss: policy_loss_fwd_bwd over the same draws packed (~4.7e5 tokens).
      sample_no_replace: the same draws without replacement (per-slot keys and
      a radix select), padded; note_use: the usage update of 256 draws;
      loss_seq_ratio, loss_asymre: the objective variants over the loss's
      tokens (12 B per token: logp, old_logp or seq id read, dlogp written);
      group_advantage: advantages of all 10^6 records in groups of 8 (4 B
      reward read + 4 B advantage written per record, 4 B per group offset);
      push: FIFO insertion of 1024 rollouts (16 B per token: tokens and
      behaviour log-probs read and written, 40 B per record).
    Algorithmic bytes: gather = 4 B/record reward scan + 4 B per positive slot
    + 20 B record metadata per draw + 8 B read per gathered token + 12 B
    written per padded position (without replacement: 8 B per record key in
    place of the reward scan); loss = 16 B per token (logp, old_logp,
    seq_of_token read, dlogp written) + 8 B per sequence."""
    import torch

    import paper_2604_08706_amd as rbp
    from paper_2604_08706_amd import workloads as wlm

    dev = "cuda"
    wl = wlm.WORKLOADS["stress"]
    tab = wlm.record_table(wl, 3)
    n = len(tab.length)
    total = int(tab.length.sum())
    tok = wlm.arena_tokens(total, wl.V, 3, device=dev)
    old = wlm.normal(total, 1.0, 4, device=dev)
    adv = wlm.normal(n, 1.0, 5, device=dev)
    keep = (torch.from_numpy(tab.arena_off).to(dev),
            torch.from_numpy(tab.length.astype(np.int32)).to(dev),
            torch.from_numpy(tab.reward).to(dev), adv, torch.from_numpy(tab.version).to(dev))
    rec = rbp.make_records(n, n, 0, *keep, tok, old)
    p_q32 = int(wl.p_pos * 2.0 ** 32)  # floor(p_pos * 2^32), the sampler's coin threshold
    n_pos = int((tab.reward > 0).sum())
    ws = rbp.workspace(rbp.RBP_OP_SAMPLE_GATHER, n)

    def cfg(step, layout, **kw):
        return rbp.make_sample_cfg(rbp.RB_POS_MIX, layout, 3, step, wl.n_draw, p_pos_q32=p_q32,
                                   cur_version=tab.cur_version, **kw)

    c_pad = cfg(0, rbp.RB_LAYOUT_PADDED, l_max=wl.l_max)
    out = rbp.alloc_batch(c_pad)
    for k in range(3):
        rbp.rb_sample_gather(rec, cfg(100 + k, rbp.RB_LAYOUT_PADDED, l_max=wl.l_max), out, ws)
    cfgs = [cfg(i, rbp.RB_LAYOUT_PADDED, l_max=wl.l_max) for i in range(iters)]
    # The calls take less GPU time than the host needs to issue them: a spin
    # kernel ahead of the timed region lets all of them queue, so the events
    # measure the GPU executing them back to back.
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for c in cfgs:
        rbp.rb_sample_gather(rec, c, out, ws)
    b.record()
    torch.cuda.synchronize()
    g_ms = a.elapsed_time(b) / iters
    n_tok = []  # valid tokens per call, from an untimed repeat (draws depend on the step only)
    for c in cfgs:
        rbp.rb_sample_gather(rec, c, out, ws)
        n_tok.append(int(out["n_tokens"].item()))
    g_bytes = float(np.mean([4 * n + 4 * n_pos + 20 * wl.n_draw + 8 * v
                             + 12 * wl.n_draw * wl.l_max for v in n_tok]))
    g_rate = g_bytes / (g_ms / 1e3)

    # without replacement: radix select over the 10^6 per-slot keys, same
    # layout; then the usage update of the drawn records
    nr = [rbp.make_sample_cfg(rbp.RB_NO_REPLACE, rbp.RB_LAYOUT_PADDED, 3, i, wl.n_draw,
                              cur_version=tab.cur_version, l_max=wl.l_max) for i in range(iters)]
    for c in nr[:3]:
        rbp.rb_sample_gather(rec, c, out, ws)
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for c in nr:
        rbp.rb_sample_gather(rec, c, out, ws)
    b.record()
    torch.cuda.synchronize()
    nr_ms = a.elapsed_time(b) / iters
    nr_tok = []
    for c in nr:
        rbp.rb_sample_gather(rec, c, out, ws)
        nr_tok.append(int(out["n_tokens"].item()))
    nr_bytes = float(np.mean([8 * n + 20 * wl.n_draw + 8 * v + 12 * wl.n_draw * wl.l_max
                              for v in nr_tok]))
    uses = torch.zeros(n, dtype=torch.int32, device=dev)
    last = torch.full((n,), -1, dtype=torch.int64, device=dev)
    since = torch.empty(wl.n_draw, dtype=torch.int32, device=dev)
    ws_u = rbp.workspace(rbp.RBP_OP_NOTE_USE, n)
    rbp.rb_note_use(out["idx"], 0, n, 0, uses, last, since, ws_u)
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for i in range(iters):
        rbp.rb_note_use(out["idx"], 0, n, i + 1, uses, last, since, ws_u)
    b.record()
    torch.cuda.synchronize()
    u_ms = a.elapsed_time(b) / iters

    # loss over the draws packed (one micro-batch holding every drawn token)
    c_pk = cfg(0, rbp.RB_LAYOUT_PACKED, max_tokens=wl.n_draw * wl.l_max)
    pk = rbp.alloc_batch(c_pk)
    rbp.rb_sample_gather(rec, c_pk, pk, ws)
    T = int(pk["n_tokens"].item())
    old_t = pk["old_logp"][:T]
    logp = old_t + wlm.normal(T, 0.05, 6, device=dev)
    seq = pk["seq_of_token"][:T]
    dlogp = torch.empty(T, device=dev)
    loss = torch.zeros(1, device=dev)
    stats = torch.zeros(4, device=dev)
    ws_l = rbp.workspace(rbp.RBP_OP_LOSS, T)
    for _ in range(3):
        rbp.policy_loss_fwd_bwd(logp, old_t, seq, pk["adv"], pk["len"], wl.n_draw, loss, dlogp,
                                stats, ws_l)
    torch.cuda.synchronize()
    torch.cuda._sleep(20_000_000)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(iters):
        rbp.policy_loss_fwd_bwd(logp, old_t, seq, pk["adv"], pk["len"], wl.n_draw, loss, dlogp,
                                stats, ws_l)
    b.record()
    torch.cuda.synchronize()
    l_ms = a.elapsed_time(b) / iters
    l_bytes = 16 * T + 8 * wl.n_draw

    def timed(fn):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        torch.cuda._sleep(20_000_000)
        ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ea.record()
        for _ in range(iters):
            fn()
        eb.record()
        torch.cuda.synchronize()
        return ea.elapsed_time(eb) / iters

    # the objective variants over the same tokens: whole-sequence ratio (the
    # draws as complete sequences) and AsymRE (stored coefficients)
    ws_s = rbp.workspace(rbp.RBP_OP_LOSS_SEQ, wl.n_draw)
    s_ms = timed(lambda: rbp.policy_loss_seq_fwd_bwd(logp, old_t, pk["cu_seqlens"], pk["adv"],
                                                     wl.n_draw, loss, dlogp, stats, ws_s))
    s_bytes = 12 * T + 8 * wl.n_draw
    st2 = torch.zeros(2, device=dev)
    a_ms = timed(lambda: rbp.policy_asymre_fwd_bwd(logp, seq, pk["adv"], wl.n_draw, loss, dlogp,
                                                   st2, ws_l))
    a_bytes = 12 * T + 4 * wl.n_draw

    # group advantages of every record of the buffer (10^6 rewards, groups of 8)
    rew_all = torch.from_numpy(tab.reward).to(dev)
    goff_all = torch.from_numpy(tab.group_off).to(dev)
    adv_all = torch.empty(n, device=dev)
    v_ms = timed(lambda: rbp.rb_group_advantage(rew_all, goff_all, adv_all))
    v_bytes = 8 * n + 4 * (len(tab.group_off))

    # FIFO insertion of 128 groups of 8 rollouts (the stress length mix) into
    # a 65536-row ring with 8192 arena tokens per row
    ring = rbp.make_ring(65536, 8192, device=dev)
    n_new = 1024
    lens = pk["len"].repeat(n_new // wl.n_draw + 1)[:n_new].contiguous()
    src = torch.zeros(n_new, dtype=torch.int64, device=dev)
    src[1:] = torch.cumsum(lens[:-1].long(), 0)
    tot = int(lens.sum().item())
    new_tok = torch.randint(0, wl.V, (tot,), dtype=torch.int32, device=dev)
    new_old = torch.randn(tot, device=dev)
    goff = torch.arange(0, n_new + 1, 8, dtype=torch.int32, device=dev)
    rew = (torch.rand(n_new, device=dev) < 0.4).float()
    p_ms = timed(lambda: rbp.rb_push(ring, goff, lens, src, rew, 1, new_tok, new_old))
    p_bytes = 16 * tot + 40 * n_new
    del tok, old, keep, rec, ring, rew_all, goff_all, adv_all
    torch.cuda.empty_cache()
    return {
        "workload": "stress: 10^6 records, 256 positive-mixture draws (p_pos 0.5), "
                    "log-normal lengths capped at 8192",
        "sample_gather": {"layout": "padded [256, 8192]", "ms": round(g_ms, 4),
                          "tokens": int(np.mean(n_tok)),
                          "bytes": int(g_bytes),
                          "GB/s": round(g_rate / 1e9, 1),
                          "frac_hbm": round(g_rate / PEAK_HBM, 4)},
        "sample_no_replace": {"layout": "padded [256, 8192]", "ms": round(nr_ms, 4),
                              "tokens": int(np.mean(nr_tok)), "bytes": int(nr_bytes),
                              "GB/s": round(nr_bytes / (nr_ms / 1e3) / 1e9, 1),
                              "frac_hbm": round(nr_bytes / (nr_ms / 1e3) / PEAK_HBM, 4)},
        "note_use": {"draws": wl.n_draw, "ms": round(u_ms, 4)},
        "loss_seq_ratio": {"tokens": T, "ms": round(s_ms, 4), "bytes": s_bytes,
                           "GB/s": round(s_bytes / (s_ms / 1e3) / 1e9, 1)},
        "loss_asymre": {"tokens": T, "ms": round(a_ms, 4), "bytes": a_bytes,
                        "GB/s": round(a_bytes / (a_ms / 1e3) / 1e9, 1)},
        "group_advantage": {"records": n, "groups": len(tab.group_off) - 1,
                            "ms": round(v_ms, 4), "bytes": v_bytes,
                            "GB/s": round(v_bytes / (v_ms / 1e3) / 1e9, 1)},
        "push": {"records": n_new, "tokens": tot, "ms": round(p_ms, 4), "bytes": p_bytes,
                 "GB/s": round(p_bytes / (p_ms / 1e3) / 1e9, 1)},
        "loss": {"tokens": T, "ms": round(l_ms, 4), "bytes": l_bytes,
                 "GB/s": round(l_bytes / (l_ms / 1e3) / 1e9, 1),
                 "frac_hbm": round(l_bytes / (l_ms / 1e3) / PEAK_HBM, 4)},
    }


def cpu_baseline(wl, n_tokens, seed=0):
    """The oracle (fp64 numpy) timed on a bounded sample of the same workload:
    the buffer draw and gather, then log-probs, loss and backward over the
    first n_tokens tokens of the micro-batch at full d and V."""
    import torch

    from oracle import buffer as ob
    from oracle.advantage import group_advantage
    from oracle.grad import logprob_backward
    from oracle.logprob import logprob
    from oracle.loss import grpo_loss
    from paper_2604_08706_amd import workloads as wlm

    tab = wlm.record_table(wl, seed)
    total = int(tab.length.sum())
    tok = wlm.arena_tokens(total, wl.V, seed).numpy()
    hidden, W, _ = wlm.head(n_tokens, wl.d, wl.V, seed)
    h64 = hidden.to(torch.float64).numpy()
    W64 = W.to(torch.float64).numpy()
    t0 = time.perf_counter()
    adv = group_advantage(tab.reward, tab.group_off)
    idx = ob.sample_indices(tab.reward, ob.RB_UNIFORM, seed, 0, wl.n_draw)
    old_arena = np.zeros(total, dtype=np.float32)
    g = ob.gather(idx, tab.arena_off, tab.length, adv, tab.version, tok, old_arena, 10,
                  ob.LAYOUT_PACKED, max_tokens=n_tokens)
    y, seq = g["tokens"], g["seq_of_token"]
    logp, lse = logprob(h64, W64, y, seq)
    loss, dlogp, _ = grpo_loss(logp, logp + 0.1, seq, g["adv"], g["len"], wl.n_draw)
    logprob_backward(h64, W64, y, lse, dlogp, seq)
    dt = time.perf_counter() - t0
    threads = os.cpu_count() or 1
    try:
        import threadpoolctl

        blas = [p["num_threads"] for p in threadpoolctl.threadpool_info()
                if p.get("user_api") == "blas"]
        if blas:
            threads = max(blas)
    except ImportError:
        pass
    return {"value": n_tokens / dt, "unit": "replayed tokens/s", "cores": threads,
            "kind": "oracle",
            "sample": f"{n_tokens} tokens of one {wl.max_tokens}-token micro-batch at "
                      f"d={wl.d}, V={wl.V} (sample+gather, advantages, log-probs, loss, "
                      f"backward in fp64 numpy); {dt:.1f} s",
            "stress_sample_gather": cpu_sampler_stress()}


def cpu_sampler_stress(seed=3):
    """The oracle's positive-mixture draw and padded gather on the 10^6-record
    stress buffer (the GPU's sample_gather line in memory_bound_steps), with
    the same algorithmic bytes.  The token arena is allocated as zeros (mapped
    lazily), so only the drawn records' stretches are touched."""
    from oracle import buffer as ob
    from paper_2604_08706_amd import workloads as wlm

    wl = wlm.WORKLOADS["stress"]
    tab = wlm.record_table(wl, seed)
    n = len(tab.length)
    total = int(tab.length.sum())
    tok = np.zeros(total, dtype=np.int32)
    old = np.zeros(total, dtype=np.float32)
    p_q32 = int(wl.p_pos * 2.0 ** 32)
    t0 = time.perf_counter()
    idx = ob.sample_indices(tab.reward, ob.RB_POS_MIX, seed, 0, wl.n_draw, p_q32=p_q32)
    g = ob.gather(idx, tab.arena_off, tab.length, np.zeros(n), tab.version, tok, old,
                  tab.cur_version, ob.LAYOUT_PADDED, l_max=wl.l_max)
    dt = time.perf_counter() - t0
    n_pos = int((tab.reward > 0).sum())
    nbytes = 4 * n + 4 * n_pos + 20 * wl.n_draw + 8 * g["n_tokens"] + 12 * wl.n_draw * wl.l_max
    return {"ms": round(dt * 1e3, 1), "tokens": int(g["n_tokens"]),
            "GB/s": round(nbytes / dt / 1e9, 4), "cores": 1,
            "sample": f"{wl.n_draw} draws from {n} records, padded [{wl.n_draw}, {wl.l_max}]"}


def run_step_fused(rbp, wl, S, step, out, ex, ev0=None, accumulate=True):
    """The same step through policy_fused_fwd_bwd (forward, loss, backward and
    entropy in one call).  ev0: an event recorded at the step start; the
    phase events of the call, if any, are in ex."""
    if ev0 is not None:
        ev0.record()
    rbp.rb_group_advantage(S["rewards"], S["group_off"], S["adv_rec"])
    rbp.rb_sample_gather(S["rec"], cfg_for(rbp, wl, step), out, S["ws_sample"])
    rbp.policy_fused_fwd_bwd(S["hidden"], S["W"], out["tokens"], out["seq_of_token"],
                             out["old_logp"], out["adv"], out["len"], wl.n_draw, S["logp"],
                             S["lse"], S["entropy"], S["loss"], S["dlogp"], S["stats"], S["dh"],
                             S["dW"], S["ws_fused"], accumulate_dW=accumulate, exec=ex)


def tokens_of_steps(rbp, wl, S, out, steps):
    """Valid tokens each step's draw packs (untimed: a draw depends only on
    the seed and the step number)."""
    n = []
    for k in steps:
        rbp.rb_sample_gather(S["rec"], cfg_for(rbp, wl, k), out, S["ws_sample"])
        n.append(int(out["n_tokens"].item()))
    return n


def spread(xs):
    return {"min": round(float(np.min(xs)), 3), "median": round(float(np.median(xs)), 3),
            "max": round(float(np.max(xs)), 3)}


PHASES = ("logits", "merge", "loss", "scale", "dW", "dhidden")  # the RBP_PHASE_* order


def fused_leg(rbp, wl, S, out, first_step, steps, warmup, ws_tokens=None, entropy=True):
    """Time the single pass over `steps` sampled batches (after `warmup`),
    with the call's phase events recorded on the caller's stream.  ws_tokens:
    size the workspace for that many tokens (the call then runs in chunks).
    entropy: also compute the per-token entropy."""
    import torch

    T = S["T"]
    S["entropy"] = torch.empty(T, device="cuda") if entropy else None
    S["ws_fused"] = rbp.workspace(rbp.RBP_OP_FUSED, ws_tokens or T, wl.d, wl.V)
    for k in range(warmup):
        run_step_fused(rbp, wl, S, first_step + k, out, None)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(1 + rbp.RBP_NUM_PHASES)]
          for _ in range(steps)]
    exs = [rbp.make_exec(e[1:]) for e in ev]  # creates the events before timing
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        run_step_fused(rbp, wl, S, first_step + warmup + i, out, exs[i], ev[i][0])
    stop.record()
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    timed = range(first_step + warmup, first_step + warmup + steps)
    n_tok = tokens_of_steps(rbp, wl, S, out, timed)
    step_ms = [e[0].elapsed_time(ev[i + 1][0]) for i, e in enumerate(ev[:-1])]
    step_ms.append(ev[-1][0].elapsed_time(stop))
    # phase k ends at phase event k + 1 (event list index k + 2)
    ph = {name: float(np.mean([e[k + 1].elapsed_time(e[k + 2]) for e in ev]))
          for k, name in enumerate(PHASES)}
    call_ms = [e[1].elapsed_time(e[-1]) for e in ev]
    del S["ws_fused"]
    torch.cuda.empty_cache()
    return {"ms_total": ms_total, "n_tok": n_tok, "step_ms": step_ms, "phase_ms": ph,
            "call_ms": call_ms, "Tc": ws_tokens or T}


def four_leg(rbp, wl, S, out, first_step, steps, warmup, ws_tokens=None):
    """Time the four-call step (forward, loss, recomputing backward)."""
    import torch

    T = S["T"]
    ws_bwd = rbp.workspace(rbp.RBP_OP_LOGPROB_BWD, ws_tokens or T, wl.d, wl.V)
    for k in range(warmup):
        run_step(rbp, wl, S, first_step + k, out, ws_bwd=ws_bwd)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        run_step(rbp, wl, S, first_step + warmup + i, out, ev[i], ws_bwd=ws_bwd)
    stop.record()
    torch.cuda.synchronize()
    ms_total = start.elapsed_time(stop)
    n_tok = tokens_of_steps(rbp, wl, S, out, range(first_step + warmup,
                                                   first_step + warmup + steps))
    step_ms = [e[0].elapsed_time(ev[i + 1][0]) for i, e in enumerate(ev[:-1])]
    step_ms.append(ev[-1][0].elapsed_time(stop))
    ph = {"fwd": float(np.mean([e[1].elapsed_time(e[2]) for e in ev])),
          "loss": float(np.mean([e[2].elapsed_time(e[3]) for e in ev])),
          "bwd": float(np.mean([e[3].elapsed_time(e[4]) for e in ev]))}
    del ws_bwd
    torch.cuda.empty_cache()
    return {"ms_total": ms_total, "n_tok": n_tok, "step_ms": step_ms, "phase_ms": ph,
            "Tc": ws_tokens or T}


def main():
    args = parse()
    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib)
        return
    if args.blas_probe:
        blas_probe()
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU "
              "data-parallel path is described in the design notes, not implemented", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2604_08706_amd as rbp
    from paper_2604_08706_amd import workloads as wlm

    wl = wlm.WORKLOADS[args.workload]
    if wl.layout != "packed":
        raise SystemExit("bench workload must use the packed layout")
    S = setup(wl)
    T = S["T"]
    K, Wm = args.steps, args.warmup
    n_legs = 2 + (0 if args.no_four_call else 1) + (0 if args.no_bounded else 2)
    align_old_logp(rbp, wl, S, range(n_legs * (K + Wm)), wl.noise_sd)
    out = rbp.alloc_batch(cfg_for(rbp, wl, 0))
    dV = wl.d * wl.V
    prod_flop = 2.0 * T * dV  # one product over the micro-batch (the tail tokens pad to 0)

    # headline: the single pass
    t_wall = time.perf_counter()
    f = fused_leg(rbp, wl, S, out, 0, K, Wm)
    t_wall = time.perf_counter() - t_wall
    tok = float(np.sum(f["n_tok"]))
    tok_s = tok / (f["ms_total"] / 1e3)
    frac = tok_s * 6 * dV / PEAK_BF16
    ph = f["phase_ms"]
    # the three products; the dW and dhidden phases each hold a main launch,
    # a launch of the last round's K halves and the small kernel that adds them
    products = {k: ph[k] for k in PRODUCTS}
    dom = max(products, key=products.get)
    dom_ms = products[dom]
    tb = traffic_bytes(dom)
    rec = {
        "metric": "replayed tokens/sec (fwd+bwd logprob+loss) at 7B shape; % bf16 MFMA peak",
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": round(f["ms_total"] / K, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; Qwen2.5-7B-shaped LM head, log-normal rollout lengths)",
        "config": {"workload": f"{wl.name}: packed micro-batch of {T} replayed tokens, "
                               f"d={wl.d}, V={wl.V}, buffer {wl.n_records} records; "
                               "single-pass entry policy_fused_fwd_bwd (one chunk)",
                   "tokens_per_step_mean": round(tok / K, 1), "d": wl.d, "V": wl.V},
        "mfma_peak_frac_6dV": round(frac, 4),
        "step_ms": spread(f["step_ms"]),
        "call_ms": spread(f["call_ms"]),
        "phase_ms": {k: round(v, 3) for k, v in ph.items()},
        "product_frac": {k: round(prod_flop / (v / 1e3) / PEAK_BF16, 4)
                         for k, v in products.items()},
        "roofline": {
            "kernel": PRODUCTS[dom],
            "bound": "mfma",
            "achieved": round(prod_flop / (dom_ms / 1e3) / 1e12, 2),
            "peak": PEAK_BF16 / 1e12,
            "unit": "TFLOP/s",
            "frac": round(prod_flop / (dom_ms / 1e3) / PEAK_BF16, 4),
            "traffic": tb,
        },
        "wall_s_timed": round(t_wall, 3),
    }
    step0 = K + Wm
    if not args.no_four_call:
        g = four_leg(rbp, wl, S, out, step0, K, Wm)
        step0 += K + Wm
        g_tok_s = float(np.sum(g["n_tok"])) / (g["ms_total"] / 1e3)
        g_bwd = g["phase_ms"]["bwd"]
        rec["four_call"] = {
            "entries": "policy_logprob_fwd + policy_loss_fwd_bwd + policy_logprob_bwd "
                       "(the forward keeps logits in registers; the backward recomputes them)",
            "tokens_per_s": round(g_tok_s, 1),
            "ms_per_step": round(g["ms_total"] / K, 3),
            "mfma_peak_frac_6dV": round(g_tok_s * 6 * dV / PEAK_BF16, 4),
            "mfma_peak_frac_8dV_executed": round(g_tok_s * 8 * dV / PEAK_BF16, 4),
            "step_ms": spread(g["step_ms"]),
            "phase_ms": {k: round(v, 3) for k, v in g["phase_ms"].items()},
            "fwd_frac": round(prod_flop / (g["phase_ms"]["fwd"] / 1e3) / PEAK_BF16, 4),
            "bwd_frac_4dV": round(2 * prod_flop / (g_bwd / 1e3) / PEAK_BF16, 4),
        }
    if not args.no_bounded:
        Tc = args.bounded_tokens
        bf = fused_leg(rbp, wl, S, out, step0, K, Wm, ws_tokens=Tc)
        step0 += K + Wm
        bg = four_leg(rbp, wl, S, out, step0, K, Wm, ws_tokens=Tc)
        step0 += K + Wm
        b_tok = float(np.sum(bf["n_tok"])) / (bf["ms_total"] / 1e3)
        g_tok = float(np.sum(bg["n_tok"])) / (bg["ms_total"] / 1e3)
        rec["bounded_workspace"] = {
            "chunk_tokens": Tc,
            "single_pass": {
                "workspace_bytes": rbp.rbp_workspace_bytes(rbp.RBP_OP_FUSED, Tc, wl.d, wl.V),
                "tokens_per_s": round(b_tok, 1), "ms_per_step": round(bf["ms_total"] / K, 3),
                "mfma_peak_frac_6dV": round(b_tok * 6 * dV / PEAK_BF16, 4),
                # the phase events of a chunked call are those of its last chunk
                "phase_ms_last_chunk": {k: round(v, 3) for k, v in bf["phase_ms"].items()}},
            "four_call": {
                "workspace_bytes": rbp.rbp_workspace_bytes(rbp.RBP_OP_LOGPROB_BWD, Tc, wl.d,
                                                           wl.V),
                "tokens_per_s": round(g_tok, 1), "ms_per_step": round(bg["ms_total"] / K, 3),
                "mfma_peak_frac_6dV": round(g_tok * 6 * dV / PEAK_BF16, 4),
                "phase_ms": {k: round(v, 3) for k, v in bg["phase_ms"].items()}},
        }
    if not args.no_aux:
        rec["memory_bound_steps"] = aux_stress()
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(wl, args.cpu_tokens)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
