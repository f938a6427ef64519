"""ctypes binding of librbpolicy.so (see include/rbpolicy.h).

Argument marshalling only: every entry point checks the torch tensors it is
given (device, dtype, contiguity, size), passes raw device pointers and the
current HIP stream to the C ABI, and raises ``RbpError`` on a nonzero status.
All computation happens in the library's HIP kernels; there is no fallback.
"""

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "librbpolicy.so")

RBP_OK = 0
RBP_EINVAL = -1
RBP_EUNSUPPORTED = -2
RBP_EWORKSPACE = -3
RBP_EHIP = -4

RB_UNIFORM = 0
RB_POS_MIX = 1
RB_POS_RETAIN = 2
RB_NO_REPLACE = 3
RB_UNUSED_FIRST = 4
RB_LAYOUT_PACKED = 0
RB_LAYOUT_PADDED = 1

RBP_OP_SAMPLE_GATHER = 1
RBP_OP_LOGPROB_FWD = 2
RBP_OP_LOSS = 3
RBP_OP_LOGPROB_BWD = 4
RBP_OP_LOSS_SEQ = 5
RBP_OP_FUSED = 6
RBP_OP_NOTE_USE = 7

RBP_PHASE_START = 0
RBP_PHASE_LOGITS = 1
RBP_PHASE_MERGE = 2
RBP_PHASE_LOSS = 3
RBP_PHASE_SCALE = 4
RBP_PHASE_DW = 5
RBP_PHASE_DHIDDEN = 6
RBP_NUM_PHASES = 7

EXPORTED = (
    "rb_sample_gather", "rb_group_advantage", "policy_logprob_fwd",
    "policy_loss_fwd_bwd", "policy_logprob_bwd", "rbp_workspace_bytes",
    "rbp_status_string", "rbp_last_error", "policy_loss_seq_fwd_bwd", "rb_asymre_coef",
    "policy_asymre_fwd_bwd", "policy_fused_fwd_bwd", "rb_push", "rb_note_use",
    "rb_hist_accumulate", "rb_sample_gather_noalloc",
)


class RbpError(RuntimeError):
    def __init__(self, fn, status, detail):
        super().__init__(f"{fn}: status {status} ({detail})")
        self.status = status


class RbRecords(ctypes.Structure):
    _fields_ = [
        ("n_live", ctypes.c_int64), ("capacity", ctypes.c_int64), ("head", ctypes.c_int64),
        ("arena_off", ctypes.c_void_p), ("length", ctypes.c_void_p),
        ("reward", ctypes.c_void_p), ("advantage", ctypes.c_void_p),
        ("version", ctypes.c_void_p), ("arena_tokens", ctypes.c_void_p),
        ("arena_old_logp", ctypes.c_void_p), ("arena_size", ctypes.c_int64),
        ("use_count", ctypes.c_void_p),
    ]


class RbRing(ctypes.Structure):
    _fields_ = [
        ("n_live", ctypes.c_int64), ("capacity", ctypes.c_int64), ("head", ctypes.c_int64),
        ("slot_tokens", ctypes.c_int64),
        ("arena_off", ctypes.c_void_p), ("length", ctypes.c_void_p),
        ("reward", ctypes.c_void_p), ("advantage", ctypes.c_void_p),
        ("version", ctypes.c_void_p), ("use_count", ctypes.c_void_p),
        ("last_step", ctypes.c_void_p), ("arena_tokens", ctypes.c_void_p),
        ("arena_old_logp", ctypes.c_void_p), ("replay_hist", ctypes.c_void_p),
        ("replay_bins", ctypes.c_int32), ("pad_", ctypes.c_int32),
    ]


class RbSampleCfg(ctypes.Structure):
    _fields_ = [
        ("mode", ctypes.c_int32), ("layout", ctypes.c_int32),
        ("seed", ctypes.c_uint64), ("step", ctypes.c_uint64),
        ("n_draw", ctypes.c_int64), ("p_pos_q32", ctypes.c_uint64),
        ("n_fresh", ctypes.c_int64), ("n_pos_keep", ctypes.c_int64),
        ("cur_version", ctypes.c_int32), ("pad_", ctypes.c_int32),
        ("max_tokens", ctypes.c_int64), ("token_begin", ctypes.c_int64),
        ("l_max", ctypes.c_int64),
    ]


class RbBatch(ctypes.Structure):
    _fields_ = [
        ("idx", ctypes.c_void_p), ("adv", ctypes.c_void_p), ("len", ctypes.c_void_p),
        ("age", ctypes.c_void_p), ("cu_seqlens", ctypes.c_void_p),
        ("tokens", ctypes.c_void_p), ("old_logp", ctypes.c_void_p),
        ("seq_of_token", ctypes.c_void_p), ("n_tokens", ctypes.c_void_p),
    ]


class RbpExec(ctypes.Structure):
    _fields_ = [("phase_event", ctypes.c_void_p * RBP_NUM_PHASES)]


def load_library(path=LIB_PATH):
    """Load librbpolicy.so and declare its signatures.  Raises if missing."""
    if not os.path.exists(path):
        raise ImportError(
            f"{path} is missing: build it with `python -m paper_2604_08706_amd.build` "
            "(the HIP library is required; there is no fallback path)")
    lib = ctypes.CDLL(path)
    vp, i32, i64, sz, f32 = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                             ctypes.c_size_t, ctypes.c_float)
    lib.rb_sample_gather.argtypes = [ctypes.POINTER(RbRecords), ctypes.POINTER(RbSampleCfg),
                                     ctypes.POINTER(RbBatch), vp, sz, vp]
    lib.rb_sample_gather_noalloc.argtypes = [ctypes.POINTER(RbRecords),
                                             ctypes.POINTER(RbSampleCfg),
                                             ctypes.POINTER(RbBatch), vp]
    lib.rb_group_advantage.argtypes = [vp, vp, i32, i32, f32, vp, vp]
    lib.policy_logprob_fwd.argtypes = [vp, vp, vp, vp, i64, i32, i32, vp, vp, vp, sz, vp]
    lib.policy_loss_fwd_bwd.argtypes = [vp, vp, vp, vp, vp, i64, i32, i64, f32, f32,
                                        vp, vp, vp, vp, sz, vp]
    lib.policy_logprob_bwd.argtypes = [vp, vp, vp, vp, vp, vp, i64, i32, i32, vp, vp,
                                       ctypes.c_int, vp, sz, vp]
    lib.policy_loss_seq_fwd_bwd.argtypes = [vp, vp, vp, vp, i64, i32, i64, f32, f32, vp, vp,
                                            vp, vp, sz, vp]
    lib.rb_asymre_coef.argtypes = [vp, vp, i32, f32, vp, vp]
    lib.policy_asymre_fwd_bwd.argtypes = [vp, vp, vp, i64, i32, i64, vp, vp, vp, vp, sz, vp]
    lib.policy_fused_fwd_bwd.argtypes = [vp, vp, vp, vp, vp, vp, vp, i64, i32, i32, i32, i64,
                                         f32, f32, vp, vp, vp, vp, vp, vp, vp, vp,
                                         ctypes.c_int, vp, sz, ctypes.POINTER(RbpExec), vp]
    lib.rb_push.argtypes = [ctypes.POINTER(RbRing), i32, i32, vp, vp, vp, vp, i32, vp, vp, i32,
                            f32, vp]
    lib.rb_note_use.argtypes = [vp, i64, i64, i64, i64, vp, vp, vp, vp, sz, vp]
    lib.rb_hist_accumulate.argtypes = [vp, i64, i32, i32, vp, vp]
    lib.rbp_workspace_bytes.argtypes = [ctypes.c_int, i64, i32, i32]
    lib.rbp_workspace_bytes.restype = sz
    lib.rbp_status_string.argtypes = [ctypes.c_int]
    lib.rbp_status_string.restype = ctypes.c_char_p
    lib.rbp_last_error.argtypes = []
    lib.rbp_last_error.restype = ctypes.c_char_p
    for name in ("rb_sample_gather", "rb_group_advantage", "policy_logprob_fwd",
                 "policy_loss_fwd_bwd", "policy_logprob_bwd"):
        getattr(lib, name).restype = ctypes.c_int
    return lib


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        _LIB = load_library()
    return _LIB


def _check(fn, status):
    if status != RBP_OK:
        detail = lib().rbp_last_error().decode() or lib().rbp_status_string(status).decode()
        raise RbpError(fn, status, detail)


def _dev(t, dtype, name, numel=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, needs {numel}")
    return ctypes.c_void_p(t.data_ptr())


def _opt(t, dtype, name, numel=None):
    return ctypes.c_void_p(0) if t is None else _dev(t, dtype, name, numel)


def _stream(stream=None):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _ws(ws):
    if ws is None:
        return ctypes.c_void_p(0), 0
    _dev(ws, ws.dtype, "ws")
    return ctypes.c_void_p(ws.data_ptr()), ws.numel() * ws.element_size()


def rbp_workspace_bytes(op, n, d=0, V=0):
    return int(lib().rbp_workspace_bytes(op, n, d, V))


def workspace(op, n, d=0, V=0, device="cuda"):
    """Allocate a workspace tensor for ``op`` (torch allocates, the library uses)."""
    return torch.empty(max(rbp_workspace_bytes(op, n, d, V), 1), dtype=torch.uint8,
                       device=device)


def rb_group_advantage(reward, group_off, adv, ddof=1, eps=1e-6, stream=None):
    n_groups = group_off.numel() - 1
    st = lib().rb_group_advantage(_dev(reward, torch.float32, "reward"),
                                  _dev(group_off, torch.int32, "group_off"), n_groups,
                                  ddof, eps, _dev(adv, torch.float32, "adv", reward.numel()),
                                  _stream(stream))
    _check("rb_group_advantage", st)


def make_records(n_live, capacity, head, arena_off, length, reward, advantage, version,
                 arena_tokens, arena_old_logp, use_count=None):
    """Build the host-side rb_records struct from device tensors.

    The struct keeps references to the tensors, so their memory stays
    allocated for as long as the struct is alive."""
    rec = RbRecords()
    rec._keep = (arena_off, length, reward, advantage, version, arena_tokens, arena_old_logp,
                 use_count)
    rec.use_count = _opt(use_count, torch.int32, "use_count", capacity).value
    rec.n_live, rec.capacity, rec.head = int(n_live), int(capacity), int(head)
    rec.arena_off = _dev(arena_off, torch.int64, "arena_off", capacity).value
    rec.length = _dev(length, torch.int32, "length", capacity).value
    rec.reward = _dev(reward, torch.float32, "reward", capacity).value
    rec.advantage = _dev(advantage, torch.float32, "advantage", capacity).value
    rec.version = _dev(version, torch.int32, "version", capacity).value
    rec.arena_tokens = _dev(arena_tokens, torch.int32, "arena_tokens").value
    rec.arena_old_logp = _dev(arena_old_logp, torch.float32, "arena_old_logp").value
    rec.arena_size = int(arena_tokens.numel())
    return rec


def make_sample_cfg(mode, layout, seed, step, n_draw, p_pos_q32=0, n_fresh=0, n_pos_keep=0,
                    cur_version=0, max_tokens=0, token_begin=0, l_max=0):
    cfg = RbSampleCfg()
    cfg.mode, cfg.layout = int(mode), int(layout)
    cfg.seed, cfg.step = int(seed), int(step)
    cfg.n_draw, cfg.p_pos_q32 = int(n_draw), int(p_pos_q32)
    cfg.n_fresh, cfg.n_pos_keep = int(n_fresh), int(n_pos_keep)
    cfg.cur_version = int(cur_version)
    cfg.max_tokens, cfg.token_begin, cfg.l_max = int(max_tokens), int(token_begin), int(l_max)
    return cfg


def alloc_batch(cfg, device="cuda"):
    """Allocate the output tensors of rb_sample_gather for ``cfg``."""
    n = cfg.n_draw
    width = cfg.max_tokens if cfg.layout == RB_LAYOUT_PACKED else n * cfg.l_max
    i32, f32 = torch.int32, torch.float32
    return {
        "idx": torch.empty(n, dtype=i32, device=device),
        "adv": torch.empty(n, dtype=f32, device=device),
        "len": torch.empty(n, dtype=i32, device=device),
        "age": torch.empty(n, dtype=i32, device=device),
        "cu_seqlens": torch.empty(n + 1, dtype=i32, device=device),
        "tokens": torch.empty(width, dtype=i32, device=device),
        "old_logp": torch.empty(width, dtype=f32, device=device),
        "seq_of_token": torch.empty(width, dtype=i32, device=device),
        "n_tokens": torch.empty(1, dtype=torch.int64, device=device),
    }


def _batch(cfg, out):
    n = cfg.n_draw
    width = cfg.max_tokens if cfg.layout == RB_LAYOUT_PACKED else n * cfg.l_max
    b = RbBatch()
    b.idx = _dev(out["idx"], torch.int32, "idx", n).value
    b.adv = _dev(out["adv"], torch.float32, "adv", n).value
    b.len = _dev(out["len"], torch.int32, "len", n).value
    b.age = _dev(out["age"], torch.int32, "age", n).value
    b.cu_seqlens = _dev(out["cu_seqlens"], torch.int32, "cu_seqlens", n + 1).value
    b.tokens = _dev(out["tokens"], torch.int32, "tokens", width).value
    b.old_logp = _dev(out["old_logp"], torch.float32, "old_logp", width).value
    b.seq_of_token = _dev(out["seq_of_token"], torch.int32, "seq_of_token", width).value
    b.n_tokens = _dev(out["n_tokens"], torch.int64, "n_tokens", 1).value
    return b


def rb_sample_gather(rec, cfg, out, ws, stream=None):
    b = _batch(cfg, out)
    wsp, wsb = _ws(ws)
    st = lib().rb_sample_gather(ctypes.byref(rec), ctypes.byref(cfg), ctypes.byref(b), wsp,
                                wsb, _stream(stream))
    _check("rb_sample_gather", st)


def rb_sample_gather_noalloc(rec, cfg, out, stream=None):
    """rb_sample_gather with the library's static per-GPU scratch as its
    workspace (no workspace tensor; calls on one GPU must not overlap)."""
    b = _batch(cfg, out)
    st = lib().rb_sample_gather_noalloc(ctypes.byref(rec), ctypes.byref(cfg), ctypes.byref(b),
                                        _stream(stream))
    _check("rb_sample_gather_noalloc", st)


def _bf16_bits(t, name, numel):
    _dev(t, torch.bfloat16, name, numel)
    return ctypes.c_void_p(t.data_ptr())


def policy_logprob_fwd(hidden, W, tokens, seq_of_token, logp, lse, ws, stream=None):
    T, d = hidden.shape
    V = W.shape[0]
    if W.shape[1] != d:
        raise ValueError("hidden and W disagree on d")
    wsp, wsb = _ws(ws)
    st = lib().policy_logprob_fwd(_bf16_bits(hidden, "hidden", T * d), _bf16_bits(W, "W", V * d),
                                  _dev(tokens, torch.int32, "tokens", T),
                                  _opt(seq_of_token, torch.int32, "seq_of_token", T), T, d, V,
                                  _dev(logp, torch.float32, "logp", T),
                                  _dev(lse, torch.float32, "lse", T), wsp, wsb, _stream(stream))
    _check("policy_logprob_fwd", st)


def policy_loss_fwd_bwd(logp, old_logp, seq_of_token, adv, seq_len, n_seq_total, loss_accum,
                        dlogp, stats, ws, eps_low=0.2, eps_high=0.2, stream=None):
    T = logp.numel()
    B = adv.numel()
    wsp, wsb = _ws(ws)
    st = lib().policy_loss_fwd_bwd(_dev(logp, torch.float32, "logp", T),
                                   _dev(old_logp, torch.float32, "old_logp", T),
                                   _dev(seq_of_token, torch.int32, "seq_of_token", T),
                                   _dev(adv, torch.float32, "adv", B),
                                   _dev(seq_len, torch.int32, "seq_len", B), T, B,
                                   int(n_seq_total), eps_low, eps_high,
                                   _dev(loss_accum, torch.float32, "loss_accum", 1),
                                   _dev(dlogp, torch.float32, "dlogp", T),
                                   _dev(stats, torch.float32, "stats", 4), wsp, wsb,
                                   _stream(stream))
    _check("policy_loss_fwd_bwd", st)


def policy_loss_seq_fwd_bwd(logp, old_logp, cu_seqlens, adv, n_seq_total, loss_accum, dlogp,
                            stats, ws, eps_low=0.2, eps_high=0.2, stream=None):
    T = logp.numel()
    B = adv.numel()
    wsp, wsb = _ws(ws)
    st = lib().policy_loss_seq_fwd_bwd(_dev(logp, torch.float32, "logp", T),
                                       _dev(old_logp, torch.float32, "old_logp", T),
                                       _dev(cu_seqlens, torch.int32, "cu_seqlens", B + 1),
                                       _dev(adv, torch.float32, "adv", B), T, B,
                                       int(n_seq_total), eps_low, eps_high,
                                       _dev(loss_accum, torch.float32, "loss_accum", 1),
                                       _dev(dlogp, torch.float32, "dlogp", T),
                                       _dev(stats, torch.float32, "stats", 4), wsp, wsb,
                                       _stream(stream))
    _check("policy_loss_seq_fwd_bwd", st)


def rb_asymre_coef(reward, group_off, coef, delta_v=-0.1, stream=None):
    n_groups = group_off.numel() - 1
    st = lib().rb_asymre_coef(_dev(reward, torch.float32, "reward"),
                              _dev(group_off, torch.int32, "group_off"), n_groups,
                              float(delta_v), _dev(coef, torch.float32, "coef", reward.numel()),
                              _stream(stream))
    _check("rb_asymre_coef", st)


def policy_asymre_fwd_bwd(logp, seq_of_token, coef, n_seq_total, loss_accum, dlogp, stats, ws,
                          stream=None):
    T = logp.numel()
    B = coef.numel()
    wsp, wsb = _ws(ws)
    st = lib().policy_asymre_fwd_bwd(_dev(logp, torch.float32, "logp", T),
                                     _dev(seq_of_token, torch.int32, "seq_of_token", T),
                                     _dev(coef, torch.float32, "coef", B), T, B,
                                     int(n_seq_total),
                                     _dev(loss_accum, torch.float32, "loss_accum", 1),
                                     _dev(dlogp, torch.float32, "dlogp", T),
                                     _dev(stats, torch.float32, "stats", 2), wsp, wsb,
                                     _stream(stream))
    _check("policy_asymre_fwd_bwd", st)


def policy_logprob_bwd(hidden, W, tokens, seq_of_token, lse, dlogp, dhidden, dW, ws,
                       accumulate_dW=False, stream=None):
    T, d = hidden.shape
    V = W.shape[0]
    wsp, wsb = _ws(ws)
    st = lib().policy_logprob_bwd(_bf16_bits(hidden, "hidden", T * d), _bf16_bits(W, "W", V * d),
                                  _dev(tokens, torch.int32, "tokens", T),
                                  _opt(seq_of_token, torch.int32, "seq_of_token", T),
                                  _dev(lse, torch.float32, "lse", T),
                                  _dev(dlogp, torch.float32, "dlogp", T), T, d, V,
                                  _dev(dhidden, torch.float32, "dhidden", T * d),
                                  _dev(dW, torch.float32, "dW", V * d),
                                  1 if accumulate_dW else 0, wsp, wsb, _stream(stream))
    _check("policy_logprob_bwd", st)


def _event_handle(ev, stream):
    # torch creates the underlying event on its first record
    if ev.cuda_event == 0:
        ev.record(stream)
    return ev.cuda_event


def make_exec(phase_events, stream=None):
    """rbp_exec from a list of RBP_NUM_PHASES torch.cuda.Events (None entries
    allowed).  The struct holds references to them, so the raw handles it
    carries stay valid while the struct is alive."""
    ex = RbpExec()
    # torch destroys an event's HIP handle when the Python object goes away
    ex._keep = list(phase_events)
    s = torch.cuda.current_stream() if stream is None else stream
    for k, ev in enumerate(phase_events):
        if ev is not None:
            ex.phase_event[k] = _event_handle(ev, s)
    return ex


def policy_fused_fwd_bwd(hidden, W, tokens, seq_of_token, old_logp, adv, seq_len, n_seq_total,
                         logp, lse, entropy, loss_accum, dlogp, stats, dhidden, dW, ws,
                         accumulate_dW=False, eps_low=0.2, eps_high=0.2, exec=None,
                         stream=None):
    """exec: None or an RbpExec of phase events (make_exec)."""
    T, d = hidden.shape
    V = W.shape[0]
    B = adv.numel()
    wsp, wsb = _ws(ws)
    st = lib().policy_fused_fwd_bwd(_bf16_bits(hidden, "hidden", T * d),
                                    _bf16_bits(W, "W", V * d),
                                    _dev(tokens, torch.int32, "tokens", T),
                                    _dev(seq_of_token, torch.int32, "seq_of_token", T),
                                    _dev(old_logp, torch.float32, "old_logp", T),
                                    _dev(adv, torch.float32, "adv", B),
                                    _dev(seq_len, torch.int32, "seq_len", B), T, d, V, B,
                                    int(n_seq_total), eps_low, eps_high,
                                    _dev(logp, torch.float32, "logp", T),
                                    _dev(lse, torch.float32, "lse", T),
                                    _opt(entropy, torch.float32, "entropy", T),
                                    _dev(loss_accum, torch.float32, "loss_accum", 1),
                                    _dev(dlogp, torch.float32, "dlogp", T),
                                    _dev(stats, torch.float32, "stats", 4),
                                    _dev(dhidden, torch.float32, "dhidden", T * d),
                                    _dev(dW, torch.float32, "dW", V * d),
                                    1 if accumulate_dW else 0, wsp, wsb,
                                    None if exec is None else ctypes.byref(exec),
                                    _stream(stream))
    _check("policy_fused_fwd_bwd", st)


def make_ring(capacity, slot_tokens, device="cuda", counters=True, replay_bins=0):
    """Allocate an empty ring record table (rb_ring) with torch; returns the
    struct, which keeps its tensors in ``ring.t``.  replay_bins > 0 (needs
    counters) adds the histogram of evicted records' replay ratios."""
    cap, st = int(capacity), int(slot_tokens)
    t = {
        "arena_off": torch.zeros(cap, dtype=torch.int64, device=device),
        "length": torch.zeros(cap, dtype=torch.int32, device=device),
        "reward": torch.zeros(cap, dtype=torch.float32, device=device),
        "advantage": torch.zeros(cap, dtype=torch.float32, device=device),
        "version": torch.zeros(cap, dtype=torch.int32, device=device),
        "use_count": torch.zeros(cap, dtype=torch.int32, device=device) if counters else None,
        "last_step": torch.full((cap,), -1, dtype=torch.int64, device=device)
        if counters else None,
        "arena_tokens": torch.zeros(cap * st, dtype=torch.int32, device=device),
        "arena_old_logp": torch.zeros(cap * st, dtype=torch.float32, device=device),
        "replay_hist": torch.zeros(int(replay_bins), dtype=torch.int64, device=device)
        if replay_bins > 0 else None,
    }
    ring = RbRing()
    ring.t = t
    ring.n_live, ring.capacity, ring.head, ring.slot_tokens = 0, cap, 0, st
    ring.replay_bins = int(replay_bins)
    for k, v in t.items():
        setattr(ring, k, 0 if v is None else v.data_ptr())
    return ring


def ring_records(ring):
    """rb_records view of a ring (for rb_sample_gather); the ring must hold at
    least one record."""
    if ring.n_live < 1:
        raise ValueError("ring_records: the ring is empty")
    t = ring.t
    return make_records(ring.n_live, ring.capacity, ring.head, t["arena_off"],
                        t["length"], t["reward"], t["advantage"], t["version"],
                        t["arena_tokens"], t["arena_old_logp"], t["use_count"])


def rb_push(ring, group_off, length, src_off, reward, version, tokens, old_logp, ddof=1,
            eps=1e-6, stream=None):
    n_new = length.numel()
    n_groups = group_off.numel() - 1
    st = lib().rb_push(ctypes.byref(ring), n_new, n_groups,
                       _dev(group_off, torch.int32, "group_off", n_groups + 1),
                       _dev(length, torch.int32, "length", n_new),
                       _dev(src_off, torch.int64, "src_off", n_new),
                       _dev(reward, torch.float32, "reward", n_new), int(version),
                       _dev(tokens, torch.int32, "tokens"),
                       _dev(old_logp, torch.float32, "old_logp"), int(ddof), float(eps),
                       _stream(stream))
    _check("rb_push", st)


def rb_note_use(idx, head, capacity, step, use_count, last_step, since, ws, stream=None):
    n = idx.numel()
    wsp, wsb = _ws(ws)
    st = lib().rb_note_use(_dev(idx, torch.int32, "idx", n), n, int(head), int(capacity),
                           int(step), _dev(use_count, torch.int32, "use_count", capacity),
                           _dev(last_step, torch.int64, "last_step", capacity),
                           _opt(since, torch.int32, "since", n), wsp, wsb, _stream(stream))
    _check("rb_note_use", st)


def rb_hist_accumulate(values, hist, lo=0, stream=None):
    n = values.numel()
    st = lib().rb_hist_accumulate(_dev(values, torch.int32, "values", n), n, int(lo),
                                  hist.numel(), _dev(hist, torch.int64, "hist"), _stream(stream))
    _check("rb_hist_accumulate", st)
