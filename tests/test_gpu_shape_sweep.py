"""Seeded sweep of shapes against the full oracle: token counts, hidden
sizes (multiples of 8) and vocabularies drawn at random, with and without a
workspace small enough to cut the batch into several token chunks (dW then
accumulates over the chunks), at both W scales.  Each case runs the four
calls (forward, then backward on a random upstream gradient) and the single
pass (with the GRPO loss), with the bars of tests/test_gpu_logprob.py and
tests/test_gpu_fused.py."""

import numpy as np
import pytest
import torch

from oracle.grad import logprob_backward
from oracle.logprob import logprob
from paper_2604_08706_amd import workloads as wlm

from gpu_util import bf16_to_f64, require_gpu, to_np
import test_gpu_fused as fused
import test_gpu_logprob as lp

pytestmark = pytest.mark.gpu


def _cases(n=24, seed=2026):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        T = int(rng.integers(1, 4001))
        d = 8 * int(rng.integers(1, 161))
        V = int(rng.integers(1, 8001))
        ws = [None, 256, 512, 768, 1280, 2048][i % 6]
        w_sd = [0.02, 1.0][(i // 6) % 2]
        out.append((T, d, V, ws, w_sd))
    return out


CASES = _cases()


@pytest.mark.parametrize("T,d,V,ws_tokens,w_sd", CASES)
def test_four_calls(T, d, V, ws_tokens, w_sd):
    rbp = require_gpu()
    print(f"[sweep] four calls T={T} d={d} V={V} ws={ws_tokens} w_sd={w_sd}", flush=True)
    hidden, W, tokens = wlm.head(T, d, V, seed=T * 7 + d + V, w_sd=w_sd)
    seq = lp._mask(T, T + 3)
    h64, W64, y = bf16_to_f64(hidden), bf16_to_f64(W), to_np(tokens)
    want_logp, want_lse = logprob(h64, W64, y, seq)
    hc, Wc, tc, sc = hidden.cuda(), W.cuda(), tokens.cuda(), torch.from_numpy(seq).cuda()
    logp, lse = lp._fwd(rbp, hc, Wc, tc, sc)
    assert np.abs(to_np(logp) - want_logp).max() < lp.LOGP_ATOL
    assert np.abs(to_np(lse) - want_lse).max() < lp.LOGP_ATOL
    dlogp = wlm.normal(T, 1.0, T + 4).numpy()
    dlogp[seq < 0] = 0.0
    want_dh, want_dW = logprob_backward(h64, W64, y, want_lse, dlogp, seq)
    dW0 = None if ws_tokens is None else wlm.normal((V, d), 1e-3, T + 5, device="cuda")
    dh, dW = lp._bwd(rbp, hc, Wc, tc, sc, lse, torch.from_numpy(dlogp).cuda(),
                     ws_tokens=ws_tokens, dW0=dW0)
    if dW0 is not None:
        want_dW = want_dW + to_np(dW0).astype(np.float64)
    lp._check_grads(to_np(dh), to_np(dW), want_dh, want_dW, y, seq)


@pytest.mark.parametrize("T,d,V,ws_tokens,w_sd", CASES)
def test_single_pass(T, d, V, ws_tokens, w_sd):
    rbp = require_gpu()
    print(f"[sweep] single pass T={T} d={d} V={V} ws={ws_tokens} w_sd={w_sd}", flush=True)
    (hidden, W, tokens, seq, lens, h64, W64, y, want_logp, want_lse, old,
     adv) = fused._case(T, d, V, w_sd, T * 11 + d + V)
    n_seq = len(lens) + 2
    dW0 = None if ws_tokens is None else wlm.normal((V, d), 1e-3, T + 6, device="cuda")
    out = fused._run(rbp, hidden.cuda(), W.cuda(), tokens.cuda(), torch.from_numpy(seq).cuda(),
                     torch.from_numpy(old).cuda(), torch.from_numpy(adv).cuda(),
                     torch.from_numpy(lens).cuda(), n_seq, ws_tokens=ws_tokens, dW0=dW0)
    fused._check(out, h64, W64, y, seq, lens, want_logp, want_lse, old, adv, n_seq,
                 dW_extra=None if dW0 is None else to_np(dW0).astype(np.float64))
