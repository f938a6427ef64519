"""Replayed-token throughput of the replay hot path on one MI355X.

One step = the whole trainer-side path over one replay micro-batch:
  rb_group_advantage  (advantages of the buffer's groups, as at insert)
  rb_sample_gather    (uniform draws from a 1024-record FIFO buffer, packed
                       into a 16384-token micro-batch)
  policy_logprob_fwd  (hidden [16384, 3584] x W [152064, 3584], bf16 MFMA,
                       online log-sum-exp)
  policy_loss_fwd_bwd (clipped GRPO, token ratios, group advantages)
  policy_logprob_bwd  (dhidden and dW, dW accumulated as over micro-batches)
Inputs are synthetic (seeded), shaped like Qwen2.5-7B's LM head and the
paper's rollout length mix; hidden states stand in for the model trunk's
output.  All inputs are resident in HBM before timing starts.

Prints one JSON line (metric: replayed tokens/s; also the fraction of the
MI355X dense bf16 MFMA peak, a roofline record for the dominant kernel, and
the CPU oracle timed on a bounded sample).
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

# HBM traffic of one policy_logprob_fwd call at the 16384-token micro-batch
# (d=3584, V=152064): FETCH_SIZE and WRITE_SIZE per dispatch from two
# rocprofv3 --pmc passes over this script, scaled by what the same counters
# read for a plain copy of known size (--copy-probe-mib: a 1 GiB copy reads
# 524302 KiB of FETCH_SIZE, factor 2.0, and 1048576 KiB of WRITE_SIZE, factor
# 1.0).  Only valid for the sources the counters were read on.
TRAFFIC_SOURCES = ("logprob.hip", "logits_epilogue.h", "gemm_core.h", "gemm_dma.h")
TRAFFIC = {
    "sources_sha256": "033a9c3d1a50806a1905286fc4f838a4dfa2ee97ad8d9719a4e9a8e7dd99744b",
    "fetch_bytes": {"logits_lse_partial_kernel": 27354198699,   # 13356542 KiB x 2.0
                    "lse_merge_kernel": 373326507},             # 182288 KiB x 2.0
    "write_bytes": {"logits_lse_partial_kernel": 117253461,     # 114505 KiB
                    "lse_merge_kernel": 264192},                # 258.0 KiB
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
                      f"backward in fp64 numpy); {dt:.1f} s"}


def run_step_fused(rbp, wl, S, step, out, ev=None):
    """The same step through policy_fused_fwd_bwd (forward, loss, backward and
    entropy in one call; keeps T x V exp(z - max) in its workspace)."""
    rbp.rb_group_advantage(S["rewards"], S["group_off"], S["adv_rec"])
    rbp.rb_sample_gather(S["rec"], cfg_for(rbp, wl, step), out, S["ws_sample"])
    if ev is not None:
        ev[0].record()
    rbp.policy_fused_fwd_bwd(S["hidden"], S["W"], out["tokens"], out["seq_of_token"],
                             out["old_logp"], out["adv"], out["len"], wl.n_draw, S["logp"],
                             S["lse"], S["entropy"], S["loss"], S["dlogp"], S["stats"], S["dh"],
                             S["dW"], S["ws_fused"], accumulate_dW=True)
    if ev is not None:
        ev[1].record()


def fused_leg(rbp, wl, S, out, first_step, steps, warmup):
    """Time the single-pass path on the same sampled batches as the main loop."""
    import torch

    S["entropy"] = torch.empty(S["T"], device="cuda")
    S["ws_fused"] = rbp.workspace(rbp.RBP_OP_FUSED, S["T"], wl.d, wl.V)
    for k in range(warmup):
        run_step_fused(rbp, wl, S, first_step + k, out)
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(2)] for _ in range(steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for i in range(steps):
        run_step_fused(rbp, wl, S, first_step + warmup + i, out, evs[i])
    stop.record()
    torch.cuda.synchronize()
    ms_step = start.elapsed_time(stop) / steps
    n_valid = int(out["n_tokens"].item())
    med = float(np.median([e[0].elapsed_time(e[1]) for e in evs]))
    dV = wl.d * wl.V
    del S["ws_fused"]
    torch.cuda.empty_cache()
    return {
        "entry": "policy_fused_fwd_bwd (stores T x V exp(z - max) in bf16; "
                 "not the headline, whose forward never materialises T x V)",
        "tokens_per_s": round(n_valid / (ms_step / 1e3), 1),
        "ms_per_step": round(ms_step, 3),
        "median_ms_fwd_loss_bwd": round(med, 3),
        "tokens_per_s_median_fwd_loss_bwd": round(n_valid / (med / 1e3), 1),
        "mfma_peak_frac_6dV": round(n_valid / (ms_step / 1e3) * 6 * dV / PEAK_BF16, 4),
        "steps": steps,
        "warmup": warmup,
    }


def main():
    args = parse()
    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU "
              "data-parallel path is a design note, not part of this build", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2604_08706_amd as rbp
    from paper_2604_08706_amd import workloads as wlm

    wl = wlm.WORKLOADS[args.workload]
    if wl.layout != "packed":
        raise SystemExit("bench workload must use the packed layout")
    S = setup(wl)
    T = S["T"]
    steps = list(range((args.warmup + args.steps) * (1 if args.no_fused else 2)))
    align_old_logp(rbp, wl, S, steps, wl.noise_sd)
    cfg0 = cfg_for(rbp, wl, 0)
    out = rbp.alloc_batch(cfg0)
    for k in range(args.warmup):
        run_step(rbp, wl, S, k, out)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(args.steps)]
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_wall = time.perf_counter()
    start.record()
    for i in range(args.steps):
        run_step(rbp, wl, S, args.warmup + i, out, evs[i])
    stop.record()
    torch.cuda.synchronize()
    t_wall = time.perf_counter() - t_wall
    ms_total = start.elapsed_time(stop)
    ms_step = ms_total / args.steps
    fwd_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in evs]))
    loss_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in evs]))
    bwd_ms = float(np.mean([e[2].elapsed_time(e[3]) for e in evs]))
    n_valid = int(out["n_tokens"].item())
    # forward + loss + backward only (the sampler excluded), median over steps
    k24_ms = float(np.median([e[0].elapsed_time(e[3]) for e in evs]))
    tok_s = n_valid * args.steps / (ms_total / 1e3)
    dV = wl.d * wl.V
    frac = tok_s * 6 * dV / PEAK_BF16
    fwd_flops = 2.0 * T * dV
    rec = {
        "metric": "replayed tokens/sec (fwd+bwd logprob+loss) at 7B shape; % bf16 MFMA peak",
        "value": round(tok_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; Qwen2.5-7B-shaped LM head, log-normal rollout lengths)",
        "config": {"workload": f"{wl.name}: packed micro-batch of {T} replayed tokens, "
                               f"d={wl.d}, V={wl.V}, buffer {wl.n_records} records",
                   "tokens_per_step": n_valid, "d": wl.d, "V": wl.V},
        "mfma_peak_frac_6dV": round(frac, 4),
        "mfma_peak_frac_8dV_executed": round(tok_s * 8 * dV / PEAK_BF16, 4),
        "median_ms_fwd_loss_bwd": round(k24_ms, 3),
        "tokens_per_s_median_fwd_loss_bwd": round(n_valid / (k24_ms / 1e3), 1),
        "phase_ms": {"fwd": round(fwd_ms, 3), "loss": round(loss_ms, 3),
                     "bwd": round(bwd_ms, 3),
                     "sample+adv+rest": round(ms_step - fwd_ms - loss_ms - bwd_ms, 3)},
        "roofline": {
            "kernel": "policy_logprob_fwd (logits_lse_partial_kernel + lse_merge_kernel)",
            "bound": "mfma",
            "achieved": round(fwd_flops / (fwd_ms / 1e3) / 1e12, 2),
            "peak": PEAK_BF16 / 1e12,
            "unit": "TFLOP/s",
            "frac": round(fwd_flops / (fwd_ms / 1e3) / PEAK_BF16, 4),
            "traffic": traffic_bytes(),
        },
        "wall_s_timed": round(t_wall, 3),
    }
    if not args.no_fused:
        rec["fused_single_pass"] = fused_leg(rbp, wl, S, out, args.warmup + args.steps,
                                             args.steps, args.warmup)
    if not args.no_aux:
        rec["memory_bound_steps"] = aux_stress()
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(wl, args.cpu_tokens)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
