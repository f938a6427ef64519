"""Dense-gradient parity at the benchmark's launch configuration (T = 16384,
d = 3584, V = 152064), for the four-call path and the single pass, each in one
16384-token chunk and with a workspace for 4096-token chunks (four chunks,
dW accumulated across them; each chunk's dhidden has 224 tiles, a last round
more than half full, cut into K pieces).

Every token of a ~2048-token block of whole sequences (inside the batch, not
tile-aligned, spanning nine token tiles) carries the loss's gradient: its
sequences have nonzero advantages, every other sequence has advantage 0, so
dlogp is exactly 0 outside the block.  The oracle (fp64) then computes the
whole result from the block's rows: log-probs, loss and dlogp, dhidden, and
dW as the sum of ~1900 dense contributions through the K = 16384 reduction.
Bars: log-probs and entropy 2e-3 absolute; loss 1e-2 relative; dlogp,
dhidden, all of dW and dW's non-target rows 1e-2 relative L2."""

import numpy as np
import pytest
import torch

from oracle.grad import logprob_backward
from oracle.logprob import entropy, logprob
from oracle.loss import grpo_loss
from paper_2604_08706_amd import workloads as wlm

from gpu_util import rel_l2, require_gpu, to_np

pytestmark = pytest.mark.gpu

ATOL = 2e-3
RTOL = 1e-2
BLOCK_START, BLOCK_TOKENS = 3000, 2048


@pytest.fixture(scope="module")
def case():
    rbp = require_gpu()
    wl = wlm.WORKLOADS["head7b"]
    T, d, V = wl.max_tokens, wl.d, wl.V
    print("[dense] inputs", flush=True)
    hidden, W, tokens = wlm.head(T, d, V, seed=17, device="cuda")
    rng = np.random.default_rng(17)
    lens = []
    while sum(lens) < T:
        lens.append(int(rng.integers(20, 600)))
    lens[-1] -= sum(lens) - T
    lens = np.array(lens, dtype=np.int32)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    seq = np.repeat(np.arange(len(lens)), lens).astype(np.int32)
    seq[rng.random(T) < 0.03] = -1  # padding inside sequences
    # the block: whole sequences from the first one starting at BLOCK_START on
    first = int(np.searchsorted(starts, BLOCK_START))
    last = first
    while starts[last] + lens[last] - starts[first] < BLOCK_TOKENS:
        last += 1
    in_block = np.arange(first, last + 1)
    rows = np.arange(starts[first], starts[last] + lens[last])
    adv = np.zeros(len(lens), dtype=np.float32)
    adv[in_block] = rng.standard_normal(len(in_block)).astype(np.float32)
    W64 = W.cpu().to(torch.float64).numpy()
    h64 = hidden[torch.from_numpy(rows).cuda()].cpu().to(torch.float64).numpy()
    y = to_np(tokens)[rows]
    sq = seq[rows]
    print(f"[dense] oracle over {len(rows)} rows of {len(in_block)} sequences", flush=True)
    logp64, lse64 = logprob(h64, W64, y, sq)
    # behaviour log-probs: the oracle's plus staleness noise N(0, 0.1^2), fp32
    old = np.zeros(T, dtype=np.float32)
    old[rows] = (logp64 + rng.normal(0.0, 0.1, len(rows))).astype(np.float32)
    loss64, dlogp64, _ = grpo_loss(logp64, old[rows], sq, adv, lens, len(lens))
    ent64 = entropy(h64, W64, sq)
    dh64, dW64 = logprob_backward(h64, W64, y, lse64, dlogp64, sq)
    print("[dense] oracle done", flush=True)
    dev = {"hidden": hidden, "W": W, "tokens": tokens, "seq": torch.from_numpy(seq).cuda(),
           "old": torch.from_numpy(old).cuda(), "adv": torch.from_numpy(adv).cuda(),
           "lens": torch.from_numpy(lens).cuda()}
    want = {"rows": rows, "y": y, "logp": logp64, "lse": lse64, "loss": loss64,
            "dlogp": dlogp64, "ent": ent64, "dh": dh64, "dW": dW64,
            "n_valid": int((seq >= 0).sum())}
    yield rbp, wl, dev, want
    del dev
    torch.cuda.empty_cache()


def _check(out, want, T, V, with_entropy):
    rows = want["rows"]
    others = np.ones(T, dtype=bool)
    others[rows] = False
    logp = to_np(out["logp"])
    assert np.abs(logp[rows] - want["logp"]).max() < ATOL
    assert np.abs(to_np(out["lse"])[rows] - want["lse"]).max() < ATOL
    if with_entropy:
        assert np.abs(to_np(out["ent"])[rows] - want["ent"]).max() < ATOL
    loss = float(to_np(out["loss"])[0])
    assert abs(loss - want["loss"]) <= RTOL * abs(want["loss"])
    dl = to_np(out["dlogp"])
    assert rel_l2(dl[rows], want["dlogp"]) < RTOL
    assert np.all(dl[others] == 0.0)
    assert to_np(out["stats"])[2] == want["n_valid"]  # every unmasked token of the batch
    dh = to_np(out["dh"])
    assert rel_l2(dh[rows], want["dh"]) < RTOL
    assert np.all(dh[others] == 0.0)
    dW = out["dW"]
    target = np.zeros(V, dtype=bool)
    target[want["y"]] = True
    num = den = num_nt = den_nt = 0.0
    for v0 in range(0, V, 16384):
        v1 = min(v0 + 16384, V)
        got = dW[v0:v1].cpu().numpy().astype(np.float64)
        w = want["dW"][v0:v1]
        num += ((got - w) ** 2).sum()
        den += (w ** 2).sum()
        nt = ~target[v0:v1]
        num_nt += ((got[nt] - w[nt]) ** 2).sum()
        den_nt += (w[nt] ** 2).sum()
    print(f"[dense] rel L2 dW {np.sqrt(num / den):.2e}, non-target {np.sqrt(num_nt / den_nt):.2e}",
          flush=True)
    assert np.sqrt(num / den) < RTOL
    assert np.sqrt(num_nt / den_nt) < RTOL


@pytest.mark.parametrize("ws_tokens", [16384, 4096])
def test_dense_four_call_path(case, ws_tokens):
    rbp, wl, dev, want = case
    T, d, V = wl.max_tokens, wl.d, wl.V
    print(f"[dense] four calls, workspace for {ws_tokens} tokens", flush=True)
    out = {"logp": torch.empty(T, device="cuda"), "lse": torch.empty(T, device="cuda"),
           "dlogp": torch.empty(T, device="cuda"), "loss": torch.zeros(1, device="cuda"),
           "stats": torch.zeros(4, device="cuda"), "dh": torch.empty((T, d), device="cuda"),
           "dW": torch.empty((V, d), device="cuda")}
    rbp.policy_logprob_fwd(dev["hidden"], dev["W"], dev["tokens"], dev["seq"], out["logp"],
                           out["lse"], rbp.workspace(rbp.RBP_OP_LOGPROB_FWD, T, d, V))
    rbp.policy_loss_fwd_bwd(out["logp"], dev["old"], dev["seq"], dev["adv"], dev["lens"],
                            dev["lens"].numel(), out["loss"], out["dlogp"], out["stats"],
                            rbp.workspace(rbp.RBP_OP_LOSS, T))
    rbp.policy_logprob_bwd(dev["hidden"], dev["W"], dev["tokens"], dev["seq"], out["lse"],
                           out["dlogp"], out["dh"], out["dW"],
                           rbp.workspace(rbp.RBP_OP_LOGPROB_BWD, ws_tokens, d, V))
    torch.cuda.synchronize()
    _check(out, want, T, V, with_entropy=False)
    del out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("ws_tokens", [16384, 4096])
def test_dense_single_pass(case, ws_tokens):
    rbp, wl, dev, want = case
    T, d, V = wl.max_tokens, wl.d, wl.V
    print(f"[dense] single pass, workspace for {ws_tokens} tokens", flush=True)
    out = {"logp": torch.empty(T, device="cuda"), "lse": torch.empty(T, device="cuda"),
           "ent": torch.empty(T, device="cuda"),
           "dlogp": torch.empty(T, device="cuda"), "loss": torch.zeros(1, device="cuda"),
           "stats": torch.zeros(4, device="cuda"), "dh": torch.empty((T, d), device="cuda"),
           "dW": torch.empty((V, d), device="cuda")}
    rbp.policy_fused_fwd_bwd(dev["hidden"], dev["W"], dev["tokens"], dev["seq"], dev["old"],
                             dev["adv"], dev["lens"], dev["lens"].numel(), out["logp"],
                             out["lse"], out["ent"], out["loss"], out["dlogp"], out["stats"],
                             out["dh"], out["dW"],
                             rbp.workspace(rbp.RBP_OP_FUSED, ws_tokens, d, V))
    torch.cuda.synchronize()
    _check(out, want, T, V, with_entropy=True)
    del out
    torch.cuda.empty_cache()
