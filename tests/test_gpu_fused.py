"""GPU parity of policy_fused_fwd_bwd (forward, loss, backward and entropy in
one pass) against the oracle: logp, lse and entropy within 2e-3 absolute;
loss within 1e-2 relative; dlogp, dhidden and dW within 1e-2 relative L2."""

import numpy as np
import pytest
import torch

from oracle.grad import dW_from_rows, dhidden_rows, dz_rows, logprob_backward
from oracle.logprob import entropy, logprob, logprob_rows
from oracle.loss import grpo_loss
from paper_2604_08706_amd import workloads as wlm

from gpu_util import bf16_to_f64, rel_l2, require_gpu, to_np

pytestmark = pytest.mark.gpu

ATOL = 2e-3
RTOL = 1e-2


def _sequences(T, seed, masked=0.1, mean_len=40):
    """Packed sequences covering T tokens (ids in order), some tokens masked."""
    rng = np.random.default_rng(seed)
    lens = []
    while sum(lens) < T:
        lens.append(int(max(1, rng.poisson(mean_len))))
    lens[-1] -= sum(lens) - T
    if lens[-1] == 0:
        lens.pop()
    seq = np.repeat(np.arange(len(lens)), lens).astype(np.int32)
    seq[rng.random(T) < masked] = -1
    return seq, np.array(lens, dtype=np.int32)


def _run(rbp, hidden, W, tokens, seq, old, adv, slen, n_seq, ws_tokens=None, dW0=None,
         want_entropy=True, ex=None, loss0=0.25, eps=(0.2, 0.2)):
    T, d = hidden.shape
    V = W.shape[0]
    out = {k: torch.empty(T, device="cuda") for k in ("logp", "lse", "dlogp")}
    out["entropy"] = torch.empty(T, device="cuda") if want_entropy else None
    out["loss"] = torch.full((1,), loss0, device="cuda")
    out["stats"] = torch.zeros(4, device="cuda")
    out["dh"] = torch.empty((T, d), device="cuda")
    out["dW"] = torch.empty((V, d), device="cuda") if dW0 is None else dW0.clone()
    ws = rbp.workspace(rbp.RBP_OP_FUSED, T if ws_tokens is None else ws_tokens, d, V)
    rbp.policy_fused_fwd_bwd(hidden, W, tokens, seq, old, adv, slen, n_seq, out["logp"],
                             out["lse"], out["entropy"], out["loss"], out["dlogp"],
                             out["stats"], out["dh"], out["dW"], ws,
                             accumulate_dW=dW0 is not None, eps_low=eps[0], eps_high=eps[1],
                             exec=ex)
    torch.cuda.synchronize()
    return out


def _case(T, d, V, w_sd, seed, device="cpu"):
    hidden, W, tokens = wlm.head(T, d, V, seed=seed, w_sd=w_sd, device=device)
    seq, lens = _sequences(T, seed + 1)
    h64, W64, y = bf16_to_f64(hidden), bf16_to_f64(W), to_np(tokens)
    want_logp, want_lse = logprob(h64, W64, y, seq)
    # behaviour log-probs: the oracle's plus staleness noise, stored as fp32
    old = (want_logp + wlm.normal(T, 0.1, seed + 2).numpy()).astype(np.float32)
    adv = wlm.normal(len(lens), 1.0, seed + 3).numpy()
    return hidden, W, tokens, seq, lens, h64, W64, y, want_logp, want_lse, old, adv


def _check(out, h64, W64, y, seq, lens, want_logp, want_lse, old, adv, n_seq, loss0=0.25,
           dW_extra=None, eps=(0.2, 0.2)):
    assert np.abs(to_np(out["logp"]) - want_logp).max() < ATOL
    assert np.abs(to_np(out["lse"]) - want_lse).max() < ATOL
    if out["entropy"] is not None:
        want_H = entropy(h64, W64, seq)
        assert np.abs(to_np(out["entropy"]) - want_H).max() < ATOL
    loss, dlogp, st = grpo_loss(want_logp, old, seq, adv, lens, n_seq, eps[0], eps[1])
    assert abs(to_np(out["loss"])[0] - loss0 - loss) <= RTOL * max(abs(loss), 1e-6)
    assert rel_l2(to_np(out["dlogp"]), dlogp) < RTOL
    assert to_np(out["stats"])[2] == st[2]
    want_dh, want_dW = logprob_backward(h64, W64, y, want_lse, dlogp, seq)
    if dW_extra is not None:
        want_dW = want_dW + dW_extra
    assert rel_l2(to_np(out["dh"]), want_dh) < RTOL
    assert rel_l2(to_np(out["dW"]), want_dW) < RTOL
    assert np.all(to_np(out["dh"])[seq < 0] == 0)


SHAPES = [(1, 8, 1), (37, 8, 300), (300, 72, 1000), (513, 136, 2049), (1000, 264, 4097)]


@pytest.mark.parametrize("T,d,V", SHAPES)
@pytest.mark.parametrize("w_sd", [0.02, 1.0])
def test_fused_small_shapes(T, d, V, w_sd):
    rbp = require_gpu()
    print(f"[fused] T={T} d={d} V={V} w_sd={w_sd}", flush=True)
    (hidden, W, tokens, seq, lens, h64, W64, y, want_logp, want_lse, old,
     adv) = _case(T, d, V, w_sd, T + d + V)
    n_seq = len(lens) + 3
    out = _run(rbp, hidden.cuda(), W.cuda(), tokens.cuda(), torch.from_numpy(seq).cuda(),
               torch.from_numpy(old).cuda(), torch.from_numpy(adv).cuda(),
               torch.from_numpy(lens).cuda(), n_seq)
    _check(out, h64, W64, y, seq, lens, want_logp, want_lse, old, adv, n_seq)


def test_fused_chunks_with_dhidden_in_pieces():
    """d = 3584 with a workspace for 4096-token chunks (the bounded-workspace
    chunk at the 7B head's width): T = 8000 runs as chunks of 4096 and 3904
    tokens, dW accumulated over both.  Each chunk's dhidden has 16 x 14 = 224
    tiles, a last round more than half full on 256 compute units, cut into K
    pieces; V = 4000 keeps the full oracle cheap."""
    rbp = require_gpu()
    T, d, V = 8000, 3584, 4000
    print(f"[fused] T={T} d={d} V={V}, 4096-token chunks", flush=True)
    (hidden, W, tokens, seq, lens, h64, W64, y, want_logp, want_lse, old,
     adv) = _case(T, d, V, 0.02, 31)
    n_seq = len(lens)
    dW0 = wlm.normal((V, d), 1e-3, 32, device="cuda")
    out = _run(rbp, hidden.cuda(), W.cuda(), tokens.cuda(), torch.from_numpy(seq).cuda(),
               torch.from_numpy(old).cuda(), torch.from_numpy(adv).cuda(),
               torch.from_numpy(lens).cuda(), n_seq, ws_tokens=4096, dW0=dW0)
    _check(out, h64, W64, y, seq, lens, want_logp, want_lse, old, adv, n_seq,
           dW_extra=to_np(dW0).astype(np.float64))


@pytest.mark.parametrize("name,T", [("head05b", 700), ("head15b", 300)])
def test_fused_real_vocab_chunked_and_accumulating(name, T):
    """Real vocabulary (151936: a V tail), then 256-token chunks with dW
    accumulation and no entropy output."""
    rbp = require_gpu()
    wl = wlm.WORKLOADS[name]
    print(f"[fused] {name} T={T}", flush=True)
    (hidden, W, tokens, seq, lens, h64, W64, y, want_logp, want_lse, old,
     adv) = _case(T, wl.d, wl.V, 0.02, 21, device="cuda")
    n_seq = len(lens)
    args = (rbp, hidden, W, tokens, torch.from_numpy(seq).cuda(), torch.from_numpy(old).cuda(),
            torch.from_numpy(adv).cuda(), torch.from_numpy(lens).cuda(), n_seq)
    out = _run(*args)
    _check(out, h64, W64, y, seq, lens, want_logp, want_lse, old, adv, n_seq)
    dW0 = wlm.normal((wl.V, wl.d), 1e-4, 7, device="cuda")
    out2 = _run(*args, ws_tokens=256, dW0=dW0, want_entropy=False)
    _check(out2, h64, W64, y, seq, lens, want_logp, want_lse, old, adv, n_seq,
           dW_extra=to_np(dW0).astype(np.float64))


def test_fused_head7b_full_size_sampled_rows():
    """T = 16384, d = 3584, V = 152064 in one chunk.  Only three short
    sequences have a nonzero advantage, so dlogp, dhidden and dW involve their
    rows alone and the oracle computes them row by row."""
    rbp = require_gpu()
    wl = wlm.WORKLOADS["head7b"]
    T = 16384
    print("[fused] head7b full size", flush=True)
    hidden, W, tokens = wlm.head(T, wl.d, wl.V, seed=0, device="cuda")
    lens = np.full(T // 64, 64, dtype=np.int32)
    seq = np.repeat(np.arange(len(lens)), lens).astype(np.int32)
    live = [0, 100, len(lens) - 1]  # first, middle and last sequence
    lens[live] = [7, 9, 11]  # full lengths; their remaining tokens are masked
    rows = np.concatenate([np.arange(64 * s, 64 * s + lens[s]) for s in live])
    mask_rows = np.concatenate([np.arange(64 * s + lens[s], 64 * s + 64) for s in live])
    seq[mask_rows] = -1
    adv = np.zeros(len(lens), dtype=np.float32)
    adv[live] = [1.0, -0.7, 0.4]
    check_rows = np.concatenate([rows, [1000, 5000, 9999]])
    h64 = hidden[torch.from_numpy(check_rows).cuda()].cpu().to(torch.float64).numpy()
    W64 = bf16_to_f64(W)
    y = to_np(tokens)[check_rows]
    want_logp, want_lse = logprob_rows(h64, W64, y, range(len(check_rows)))
    rng = np.random.default_rng(1)
    old = np.full(T, -5.0, dtype=np.float32)
    old[check_rows] = (want_logp + rng.normal(0, 0.1, len(check_rows))).astype(np.float32)
    n_seq = len(lens)
    out = _run(rbp, hidden, W, tokens, torch.from_numpy(seq).cuda(),
               torch.from_numpy(old).cuda(), torch.from_numpy(adv).cuda(),
               torch.from_numpy(lens).cuda(), n_seq)
    assert np.abs(to_np(out["logp"])[check_rows] - want_logp).max() < ATOL
    assert np.abs(to_np(out["lse"])[check_rows] - want_lse).max() < ATOL
    want_H = entropy(h64, W64)
    assert np.abs(to_np(out["entropy"])[check_rows] - want_H).max() < ATOL
    for key in ("logp", "lse", "entropy"):
        assert np.all(to_np(out[key])[mask_rows] == 0), key
    k = len(rows)
    _, dl_rows, _ = grpo_loss(want_logp[:k], old[rows], seq[rows], adv, lens, n_seq)
    dl = to_np(out["dlogp"])
    assert rel_l2(dl[rows], dl_rows) < RTOL
    others = np.ones(T, dtype=bool)
    others[rows] = False
    assert np.all(dl[others] == 0)
    dh = to_np(out["dh"])
    assert np.all(dh[others] == 0)
    dz = dz_rows(h64[:k], W64, y[:k], want_lse[:k], dl_rows, range(k))
    want_dh = dhidden_rows(h64[:k], W64, y[:k], want_lse[:k], dl_rows, range(k), dz=dz)
    assert rel_l2(dh[rows], want_dh) < RTOL
    num = den = 0.0
    for v0 in range(0, wl.V, 16384):
        v1 = min(v0 + 16384, wl.V)
        want = dW_from_rows(h64[:k], W64, y[:k], want_lse[:k], dl_rows, range(k), v0, v1, dz=dz)
        got = out["dW"][v0:v1].cpu().numpy().astype(np.float64)
        num += ((got - want) ** 2).sum()
        den += (want ** 2).sum()
    assert np.sqrt(num / den) < RTOL
    del hidden, W, out
    torch.cuda.empty_cache()


def test_fused_reproducible_empty_and_bad_args():
    rbp = require_gpu()
    T, d, V = 600, 128, 3000
    (hidden, W, tokens, seq, lens, *_rest) = _case(T, d, V, 0.02, 5, device="cuda")
    old, adv = _rest[-2], _rest[-1]
    args = (rbp, hidden, W, tokens, torch.from_numpy(seq).cuda(), torch.from_numpy(old).cuda(),
            torch.from_numpy(adv).cuda(), torch.from_numpy(lens).cuda(), len(lens))
    a, b = _run(*args), _run(*args)
    for key in ("logp", "lse", "entropy", "loss", "dlogp", "stats", "dh", "dW"):
        assert torch.equal(a[key], b[key]), key
    # T = 0 zeroes dW (overwrite mode)
    dW = torch.full((V, d), 3.0, device="cuda")
    e0 = torch.empty(0, device="cuda")
    rbp.policy_fused_fwd_bwd(hidden[:0], W, tokens[:0], torch.empty(0, dtype=torch.int32,
                                                                     device="cuda"),
                             e0, args[6], args[7], len(lens), e0, e0, None,
                             torch.zeros(1, device="cuda"), e0, torch.zeros(4, device="cuda"),
                             torch.empty((0, d), device="cuda"), dW, None)
    torch.cuda.synchronize()
    assert torch.count_nonzero(dW).item() == 0
    with pytest.raises(rbp.RbpError) as e:
        rbp.policy_fused_fwd_bwd(hidden, W, tokens, args[4], args[5], args[6], args[7], len(lens),
                                 a["logp"], a["lse"], None, a["loss"], a["dlogp"], a["stats"],
                                 a["dh"], a["dW"],
                                 torch.empty(16, dtype=torch.uint8, device="cuda"))
    assert e.value.status == rbp.RBP_EWORKSPACE


def test_fused_concurrent_calls_on_two_streams():
    """Two host threads run the single pass on their own streams at once (the
    library holds no state between calls); every result must equal the same
    call made alone."""
    import threading

    rbp = require_gpu()
    T, d, V = 2048, 512, 70000
    cases = []
    for seed in (31, 32):
        (hidden, W, tokens, seq, lens, *_r) = _case(T, d, V, 0.02, seed, device="cuda")
        old, adv = _r[-2], _r[-1]
        cases.append((rbp, hidden, W, tokens, torch.from_numpy(seq).cuda(),
                      torch.from_numpy(old).cuda(), torch.from_numpy(adv).cuda(),
                      torch.from_numpy(lens).cuda(), len(lens)))
    alone = [_run(*c) for c in cases]
    results = [[None] * 3 for _ in cases]
    errors = []

    def worker(i):
        try:
            st = torch.cuda.Stream()
            with torch.cuda.stream(st):
                for k in range(3):
                    results[i][k] = _run(*cases[i])
        except Exception as e:  # reported by the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    assert not errors, errors
    for i in range(2):
        for k in range(3):
            for key in ("logp", "lse", "entropy", "dlogp", "dh", "dW"):
                assert torch.equal(results[i][k][key], alone[i][key]), (i, k, key)


def test_fused_three_chunks_with_sequences_across_chunk_boundaries():
    """T = 49152 at the 7B head with a workspace for 16384 tokens: three
    chunks, dW accumulated across them.  Four short sequences carry the only
    nonzero advantages, two of them straddling a chunk boundary, so dlogp,
    dhidden and dW involve their rows alone."""
    rbp = require_gpu()
    wl = wlm.WORKLOADS["head7b"]
    T, Tc = 3 * 16384, 16384
    print("[fused] head7b three chunks", flush=True)
    hidden, W, tokens = wlm.head(T, wl.d, wl.V, seed=5, device="cuda")
    L = 64
    lens = np.full(T // L, L, dtype=np.int32)
    seq = np.repeat(np.arange(len(lens)), lens).astype(np.int32)
    # sequences re-cut so that two of them cross the chunk boundaries
    starts = [100, Tc - 5, 2 * Tc - 9, T - 12]
    sizes = [9, 11, 17, 12]
    seq[:] = -1
    for i, (a, n) in enumerate(zip(starts, sizes)):
        seq[a:a + n] = i
    n_seq = 64
    lens = np.zeros(n_seq, dtype=np.int32)
    lens[:4] = sizes
    lens[4:] = 1  # sequences with no tokens in this batch
    adv = np.zeros(n_seq, dtype=np.float32)
    adv[:4] = [0.8, -1.1, 0.5, -0.3]
    rows = np.concatenate([np.arange(a, a + n) for a, n in zip(starts, sizes)])
    h64 = hidden[torch.from_numpy(rows).cuda()].cpu().to(torch.float64).numpy()
    W64 = bf16_to_f64(W)
    y = to_np(tokens)[rows]
    want_logp, want_lse = logprob_rows(h64, W64, y, range(len(rows)))
    rng = np.random.default_rng(2)
    old = np.zeros(T, dtype=np.float32)
    old[rows] = (want_logp + rng.normal(0, 0.1, len(rows))).astype(np.float32)
    dW0 = wlm.normal((wl.V, wl.d), 1e-4, 9, device="cuda")
    out = _run(rbp, hidden, W, tokens, torch.from_numpy(seq).cuda(), torch.from_numpy(old).cuda(),
               torch.from_numpy(adv).cuda(), torch.from_numpy(lens).cuda(), n_seq, ws_tokens=Tc,
               dW0=dW0)
    assert np.abs(to_np(out["logp"])[rows] - want_logp).max() < ATOL
    assert np.abs(to_np(out["lse"])[rows] - want_lse).max() < ATOL
    assert np.abs(to_np(out["entropy"])[rows] - entropy(h64, W64)).max() < ATOL
    _, dl_rows, _ = grpo_loss(want_logp, old[rows], seq[rows], adv, lens, n_seq)
    dl = to_np(out["dlogp"])
    assert rel_l2(dl[rows], dl_rows) < RTOL
    others = np.ones(T, dtype=bool)
    others[rows] = False
    assert np.all(dl[others] == 0) and np.all(to_np(out["dh"])[others] == 0)
    dz = dz_rows(h64, W64, y, want_lse, dl_rows, range(len(rows)))
    want_dh = dhidden_rows(h64, W64, y, want_lse, dl_rows, range(len(rows)), dz=dz)
    assert rel_l2(to_np(out["dh"])[rows], want_dh) < RTOL
    num = den = 0.0
    for v0 in range(0, wl.V, 16384):
        v1 = min(v0 + 16384, wl.V)
        want = dW_from_rows(h64, W64, y, want_lse, dl_rows, range(len(rows)), v0, v1, dz=dz)
        # the accumulated gradient alone (the initial dW would dominate a norm)
        got = (out["dW"][v0:v1].cpu().numpy().astype(np.float64)
               - dW0[v0:v1].cpu().numpy().astype(np.float64))
        num += ((got - want) ** 2).sum()
        den += (want ** 2).sum()
    assert np.sqrt(num / den) < RTOL
    del hidden, W, out, dW0
    torch.cuda.empty_cache()


def test_fused_phase_events():
    """Phase events recorded on the caller's stream bracket every phase in
    order and change no result; an rbp_exec keeps its torch events alive."""
    import gc

    rbp = require_gpu()
    T, d, V = 2048, 512, 70000
    (hidden, W, tokens, seq, lens, *_r) = _case(T, d, V, 0.02, 41, device="cuda")
    old, adv = _r[-2], _r[-1]
    args = (rbp, hidden, W, tokens, torch.from_numpy(seq).cuda(), torch.from_numpy(old).cuda(),
            torch.from_numpy(adv).cuda(), torch.from_numpy(lens).cuda(), len(lens))
    ex = rbp.make_exec([torch.cuda.Event(enable_timing=True) for _ in range(rbp.RBP_NUM_PHASES)])
    evs = ex._keep
    gc.collect()
    a = _run(*args, ex=ex)
    ms = [evs[k].elapsed_time(evs[k + 1]) for k in range(rbp.RBP_NUM_PHASES - 1)]
    assert all(m >= 0.0 for m in ms) and sum(ms) > 0.0, ms
    b = _run(*args)
    c = _run(*args, ex=rbp.make_exec(evs[:3] + [None] * 4))
    for key in ("logp", "lse", "entropy", "loss", "dlogp", "stats", "dh", "dW"):
        assert torch.equal(a[key], b[key]), key
        assert torch.equal(a[key], c[key]), key


@pytest.mark.parametrize("shift,adv_sign", [(35.0, 1.0), (-45.0, -1.0), ("mixed", 0.0),
                                            (15.0, 1.0), (-30.0, -1.0), (22.0, 1.0),
                                            (24.0, 1.0), (-37.5, -1.0), (-38.5, -1.0)])
def test_fused_tokens_off_their_reference(shift, adv_sign):
    """Tokens whose behaviour log-prob puts the reference R_t far from their
    largest logit take the re-referencing path: old = logp + 35 (ratio e^-35,
    positive advantages, so a tiny but unclipped gradient) or old = logp - 45
    (ratio e^45, negative advantages: an unclipped gradient e^45 times the
    usual).  'mixed': half the sequences shifted by +35, the rest ordinary, so
    the pass must leave the ordinary tokens' columns alone.  Shifts of +15
    and -30 keep every half tile's sums inside the range the store pass takes
    directly against R_t (q up to e^15; c_t of order e^30), so that path is
    checked far from R_t = lse_t too.  The logits here are nearly flat, so a
    half tile's sum is about e^shift / 32 (R_t = lse_t - shift, 32 half tiles
    at V = 4097): +22 / +24 put it just under / over the direct range's
    upper bound 2^28, and -37.5 / -38.5 just over / under its lower bound
    2^-60, so with the staleness noise and the spread of the logits waves
    take either form between neighbouring tokens.  Everything against the oracle at the
    usual bars; in the mixed case dhidden is also checked on each group's
    rows alone."""
    rbp = require_gpu()
    T, d, V = 700, 136, 4097
    (hidden, W, tokens, seq, lens, h64, W64, y, want_logp, want_lse, old,
     adv) = _case(T, d, V, 0.02, 53)
    rng = np.random.default_rng(54)
    B = len(lens)
    if shift == "mixed":
        shifted = rng.random(B) < 0.5
        adv = np.where(shifted, np.abs(adv), adv)
        tok_shift = np.where((seq >= 0) & shifted[np.maximum(seq, 0)], 35.0, 0.0)
    else:
        adv = adv_sign * np.abs(adv) + adv_sign * 0.1
        tok_shift = np.full(T, shift)
    old = (want_logp + tok_shift + rng.normal(0, 0.05, T)).astype(np.float32)
    print(f"[fused] off-reference tokens shift={shift}", flush=True)
    out = _run(rbp, hidden.cuda(), W.cuda(), tokens.cuda(), torch.from_numpy(seq).cuda(),
               torch.from_numpy(old).cuda(), torch.from_numpy(adv.astype(np.float32)).cuda(),
               torch.from_numpy(lens).cuda(), B, loss0=0.0)
    assert np.abs(to_np(out["logp"]) - want_logp).max() < ATOL
    assert np.abs(to_np(out["lse"]) - want_lse).max() < ATOL
    loss, dlogp, _ = grpo_loss(want_logp, old, seq, adv, lens, B)
    assert abs(to_np(out["loss"])[0] - loss) <= RTOL * abs(loss)
    assert rel_l2(to_np(out["dlogp"]), dlogp) < RTOL
    want_dh, want_dW = logprob_backward(h64, W64, y, want_lse, dlogp, seq)
    dh, dW = to_np(out["dh"]), to_np(out["dW"])
    assert np.all(np.isfinite(dh)) and np.all(np.isfinite(dW))
    assert rel_l2(dh, want_dh) < RTOL
    assert rel_l2(dW, want_dW) < RTOL
    if shift == "mixed":
        for grp in (tok_shift > 0, (tok_shift == 0) & (seq >= 0)):
            assert rel_l2(dh[grp], want_dh[grp]) < RTOL


def test_fused_infinite_behaviour_logprobs():
    """Tokens whose stored behaviour log-prob is -inf or +inf (ratio +inf or
    0) in sequences with positive advantages: the objective puts them on a
    zero-gradient branch, so dlogp, dhidden and dW stay finite and equal the
    oracle's; their references R_t = z_y - old_logp are infinite, so the
    single pass re-references their columns to their largest logits."""
    rbp = require_gpu()
    T, d, V = 300, 72, 1000
    print(f"[fused] T={T} d={d} V={V} infinite old_logp", flush=True)
    (hidden, W, tokens, seq, lens, h64, W64, y, want_logp, want_lse, old,
     adv) = _case(T, d, V, 0.02, 51)
    adv = np.abs(adv) + 0.1
    valid = np.flatnonzero(seq >= 0)
    pick = valid[np.linspace(0, len(valid) - 1, 12).astype(int)]
    old = old.copy()
    old[pick[::2]] = -np.inf
    old[pick[1::2]] = np.inf
    n_seq = len(lens)
    out = _run(rbp, hidden.cuda(), W.cuda(), tokens.cuda(), torch.from_numpy(seq).cuda(),
               torch.from_numpy(old).cuda(), torch.from_numpy(adv).cuda(),
               torch.from_numpy(lens).cuda(), n_seq)
    for k in ("logp", "lse", "entropy", "dlogp", "dh", "dW", "loss"):
        assert np.isfinite(to_np(out[k])).all(), k
    assert np.all(to_np(out["dlogp"])[pick] == 0)
    with np.errstate(over="ignore", invalid="ignore"):
        _check(out, h64, W64, y, seq, lens, want_logp, want_lse, old, adv, n_seq)
