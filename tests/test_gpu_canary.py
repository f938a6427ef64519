"""Output canaries: every entry point writes inside its outputs and workspace
only.  Each output (and the workspace) is a view into a larger device buffer
whose bytes before and after the view hold a sentinel pattern; after the call
the guard bytes are compared with the pattern on the host.  Shapes have tails
in every dimension (V not a multiple of 256, T = 1, d = 8, windows that end
inside the token stream), where a kernel's edge handling is most likely to
spill."""

import numpy as np
import pytest
import torch

from paper_2604_08706_amd import workloads as wlm

from gpu_util import DeviceRing, require_gpu

pytestmark = pytest.mark.gpu

PAD = 4096          # guard bytes on each side (a multiple of 256 keeps views aligned)
SENTINEL = 0xA5


class Guarded:
    """Views carved from sentinel-filled device buffers, checked afterwards."""

    def __init__(self):
        self.bufs = []

    def __call__(self, shape, dtype, fill=None):
        shape = (shape,) if isinstance(shape, int) else tuple(shape)
        n = int(np.prod(shape)) if shape else 1
        nbytes = n * torch.empty((), dtype=dtype).element_size()
        back = torch.full((PAD + nbytes + PAD,), SENTINEL, dtype=torch.uint8, device="cuda")
        view = back[PAD:PAD + nbytes].view(dtype).view(shape)
        if fill is not None:
            view.copy_(fill if isinstance(fill, torch.Tensor) else torch.full_like(view, fill))
        self.bufs.append((back, nbytes))
        return view

    def ws(self, nbytes):
        return self((max(int(nbytes), 1),), torch.uint8)

    def check(self, what):
        torch.cuda.synchronize()
        for i, (back, nbytes) in enumerate(self.bufs):
            h = back.cpu().numpy()
            assert np.all(h[:PAD] == SENTINEL), (what, i, "guard before")
            assert np.all(h[PAD + nbytes:] == SENTINEL), (what, i, "guard after")


# the last two run dhidden's round in K pieces (3 and 15 per tile)
SHAPES = [(1, 8, 1), (37, 8, 300), (513, 72, 4097), (300, 136, 2049), (9316, 1024, 3001),
          (4133, 3584, 9000)]


def _seq(T, seed):
    rng = np.random.default_rng(seed)
    lens = []
    while sum(lens) < T:
        lens.append(int(rng.integers(1, 40)))
    lens[-1] -= sum(lens) - T
    seq = np.repeat(np.arange(len(lens)), lens).astype(np.int32)
    seq[rng.random(T) < 0.1] = -1
    return seq, np.array(lens, dtype=np.int32)


@pytest.mark.parametrize("T,d,V", SHAPES)
def test_logprob_loss_backward_stay_inside(T, d, V):
    rbp = require_gpu()
    print(f"[canary] four calls T={T} d={d} V={V}", flush=True)
    g = Guarded()
    hidden, W, tokens = wlm.head(T, d, V, seed=T + V, device="cuda")
    seq_np, lens_np = _seq(T, 3)
    seq = torch.from_numpy(seq_np).cuda()
    B = len(lens_np)
    logp, lse = g(T, torch.float32), g(T, torch.float32)
    rbp.policy_logprob_fwd(hidden, W, tokens, seq, logp, lse,
                           g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_LOGPROB_FWD, T, d, V)))
    g.check("policy_logprob_fwd")
    old = (logp + 0.05).contiguous()
    adv = g(B, torch.float32, wlm.normal(B, 1.0, 4, device="cuda"))
    slen = g(B, torch.int32, torch.from_numpy(lens_np).cuda())
    loss, stats, dlogp = g(1, torch.float32, 0.0), g(4, torch.float32, 0.0), g(T, torch.float32)
    rbp.policy_loss_fwd_bwd(logp, old, seq, adv, slen, B, loss, dlogp, stats,
                            g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_LOSS, T)))
    g.check("policy_loss_fwd_bwd")
    dh, dW = g((T, d), torch.float32), g((V, d), torch.float32)
    for acc in (False, True):
        rbp.policy_logprob_bwd(hidden, W, tokens, seq, lse, dlogp, dh, dW,
                               g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_LOGPROB_BWD, T, d, V)),
                               accumulate_dW=acc)
        g.check(f"policy_logprob_bwd acc={acc}")
    # several chunks: a workspace for 256 tokens
    if T > 256:
        rbp.policy_logprob_bwd(hidden, W, tokens, seq, lse, dlogp, dh, dW,
                               g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_LOGPROB_BWD, 256, d, V)))
        g.check("policy_logprob_bwd chunked")


@pytest.mark.parametrize("T,d,V", SHAPES)
def test_fused_stays_inside(T, d, V):
    rbp = require_gpu()
    print(f"[canary] fused T={T} d={d} V={V}", flush=True)
    g = Guarded()
    hidden, W, tokens = wlm.head(T, d, V, seed=T + 2 * V, device="cuda")
    seq_np, lens_np = _seq(T, 5)
    B = len(lens_np)
    seq = torch.from_numpy(seq_np).cuda()
    old = wlm.normal(T, 1.0, 6, device="cuda") - 6.0
    adv = wlm.normal(B, 1.0, 7, device="cuda")
    slen = torch.from_numpy(lens_np).cuda()
    outs = [g(T, torch.float32) for _ in range(4)]  # logp, lse, entropy, dlogp
    loss, stats = g(1, torch.float32, 0.0), g(4, torch.float32, 0.0)
    dh, dW = g((T, d), torch.float32), g((V, d), torch.float32, 0.0)
    for ws_tok in (T, 256):
        ws = g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_FUSED, ws_tok, d, V))
        rbp.policy_fused_fwd_bwd(hidden, W, tokens, seq, old, adv, slen, B, outs[0], outs[1],
                                 outs[2], loss, outs[3], stats, dh, dW, ws, accumulate_dW=True)
        g.check(f"policy_fused_fwd_bwd ws_tokens={ws_tok}")


@pytest.mark.parametrize("T", [1, 37, 1000])
def test_objective_variants_stay_inside(T):
    rbp = require_gpu()
    print(f"[canary] objective variants T={T}", flush=True)
    g = Guarded()
    seq_np, lens_np = _seq(T, 9)
    B = len(lens_np)
    seq = torch.from_numpy(seq_np).cuda()
    logp = wlm.normal(T, 1.0, 10, device="cuda") - 5.0
    old = (logp + wlm.normal(T, 0.01, 11, device="cuda")).contiguous()
    # whole-sequence ratio: sequences packed by cu_seqlens
    cu = torch.from_numpy(np.concatenate([[0], np.cumsum(lens_np)]).astype(np.int32)).cuda()
    adv = wlm.normal(B, 1.0, 12, device="cuda")
    loss, stats, dlogp = g(1, torch.float32, 0.0), g(4, torch.float32, 0.0), g(T, torch.float32)
    rbp.policy_loss_seq_fwd_bwd(logp, old, cu, adv, B, loss, dlogp, stats,
                                g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_LOSS_SEQ, B)))
    g.check("policy_loss_seq_fwd_bwd")
    rew = (torch.rand(B, device="cuda") < 0.5).float()
    goff = torch.arange(0, B + 1, dtype=torch.int32, device="cuda")
    coef = g(B, torch.float32)
    rbp.rb_asymre_coef(rew, goff, coef)
    g.check("rb_asymre_coef")
    st2 = g(2, torch.float32, 0.0)
    rbp.policy_asymre_fwd_bwd(logp, seq, coef, B, loss, dlogp, st2,
                              g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_LOSS, T)))
    g.check("policy_asymre_fwd_bwd")
    adv2 = g(B, torch.float32)
    rbp.rb_group_advantage(rew, goff, adv2)
    g.check("rb_group_advantage")


def _ring(rbp, n, V, seed):
    rng = np.random.default_rng(seed)
    length = rng.integers(1, 200, n)
    off = np.concatenate([[0], np.cumsum(length)[:-1]])
    total = int(length.sum())
    return DeviceRing(rbp, length, off, (rng.random(n) < 0.4).astype(np.float32),
                      rng.standard_normal(n).astype(np.float32), rng.integers(0, 5, n),
                      rng.integers(0, V, total).astype(np.int32),
                      rng.standard_normal(total).astype(np.float32), head=n // 3,
                      capacity=n + 17)


@pytest.mark.parametrize("mode", ["uniform", "pos_mix", "pos_retain", "no_replace",
                                  "unused_first"])
@pytest.mark.parametrize("layout,n_draw,max_tokens,token_begin,l_max",
                         [("packed", 13, 777, 0, 0), ("packed", 40, 1000, 1500, 0),
                          ("packed", 1, 1, 0, 0), ("padded", 13, 0, 0, 57)])
def test_sample_gather_stays_inside(mode, layout, n_draw, max_tokens, token_begin, l_max):
    rbp = require_gpu()
    print(f"[canary] sample_gather {mode} {layout} n_draw={n_draw}", flush=True)
    n = 300
    ring = _ring(rbp, n, 1000, 13)
    if mode in ("no_replace", "unused_first"):
        use = torch.from_numpy(np.random.default_rng(2).integers(0, 3, ring.capacity)
                               .astype(np.int32)).cuda()
        rec = rbp.make_records(n, ring.capacity, n // 3, ring.t_off, ring.t_len, ring.t_rew,
                               ring.t_adv, ring.t_ver, ring.t_tok, ring.t_old, use)
    else:
        rec = ring.rec
    m = {"uniform": rbp.RB_UNIFORM, "pos_mix": rbp.RB_POS_MIX, "pos_retain": rbp.RB_POS_RETAIN,
         "no_replace": rbp.RB_NO_REPLACE, "unused_first": rbp.RB_UNUSED_FIRST}[mode]
    lay = rbp.RB_LAYOUT_PACKED if layout == "packed" else rbp.RB_LAYOUT_PADDED
    cfg = rbp.make_sample_cfg(m, lay, 7, 2, n_draw, p_pos_q32=int(0.6 * 2 ** 32),
                              n_fresh=200, n_pos_keep=50, cur_version=9,
                              max_tokens=max_tokens, token_begin=token_begin, l_max=l_max)
    width = max_tokens if lay == rbp.RB_LAYOUT_PACKED else n_draw * l_max
    g = Guarded()
    out = {"idx": g(n_draw, torch.int32), "adv": g(n_draw, torch.float32),
           "len": g(n_draw, torch.int32), "age": g(n_draw, torch.int32),
           "cu_seqlens": g(n_draw + 1, torch.int32), "tokens": g(width, torch.int32),
           "old_logp": g(width, torch.float32), "seq_of_token": g(width, torch.int32),
           "n_tokens": g(1, torch.int64)}
    rbp.rb_sample_gather(rec, cfg, out, g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_SAMPLE_GATHER,
                                                                     ring.capacity)))
    g.check(f"rb_sample_gather {mode} {layout}")


def test_buffer_maintenance_stays_inside():
    rbp = require_gpu()
    print("[canary] note_use, hist, push", flush=True)
    g = Guarded()
    cap, n_live, head = 500, 430, 123
    idx = torch.from_numpy(np.random.default_rng(4).integers(0, n_live, 37).astype(np.int32)).cuda()
    uses = g(cap, torch.int32, 0)
    last = g(cap, torch.int64, -1)
    since = g(37, torch.int32)
    rbp.rb_note_use(idx, head, cap, 5, uses, last, since,
                    g.ws(rbp.rbp_workspace_bytes(rbp.RBP_OP_NOTE_USE, cap)))
    g.check("rb_note_use")
    vals = torch.from_numpy(np.random.default_rng(5).integers(-3, 40, 1001)
                            .astype(np.int32)).cuda()
    hist = g(17, torch.int64, 0)
    rbp.rb_hist_accumulate(vals, hist, lo=-1)
    g.check("rb_hist_accumulate")
    # a push into a ring whose arrays are all guarded views
    ring = rbp.make_ring(40, 6, replay_bins=5)
    for k in list(ring.t):
        t = ring.t[k]
        if t is None:
            continue
        v = g(t.shape, t.dtype, t)
        ring.t[k] = v
        setattr(ring, k, v.data_ptr())
    lens = torch.tensor([3, 9, 1, 6, 7] * 6, dtype=torch.int32, device="cuda")
    src = torch.zeros(30, dtype=torch.int64, device="cuda")
    src[1:] = torch.cumsum(lens[:-1].long(), 0)
    tot = int(lens.sum().item())
    goff = torch.tensor([0, 10, 20, 30], dtype=torch.int32, device="cuda")
    for v in range(3):  # the second and third pushes evict
        rbp.rb_push(ring, goff, lens, src, (torch.rand(30, device="cuda") < 0.5).float(), v,
                    torch.randint(0, 100, (tot,), dtype=torch.int32, device="cuda"),
                    torch.randn(tot, device="cuda"))
        g.check(f"rb_push {v}")
