"""MI355X (gfx950) replay-buffer policy-gradient hot path.

Trainer-side path of experience-replay RL for LLMs (arXiv 2604.08706): seeded
replay-buffer sample-and-gather, per-token policy log-probabilities from final
hidden states and the LM head (bf16 MFMA with an online log-sum-exp), the
clipped importance-weighted GRPO loss with group advantages, and the backward
to the hidden states and the LM head.  All compute is in librbpolicy.so
(hand-written HIP); this package is a thin ctypes binding over its C ABI
(include/rbpolicy.h) and uses torch only for device memory and streams.
"""

from ._binding import (  # noqa: F401
    EXPORTED,
    LIB_PATH,
    RB_LAYOUT_PACKED,
    RB_LAYOUT_PADDED,
    RB_POS_MIX,
    RB_NO_REPLACE,
    RB_POS_RETAIN,
    RB_UNUSED_FIRST,
    RB_UNIFORM,
    RBP_EHIP,
    RBP_EINVAL,
    RBP_EUNSUPPORTED,
    RBP_EWORKSPACE,
    RBP_OK,
    RBP_OP_LOGPROB_BWD,
    RBP_OP_LOGPROB_FWD,
    RBP_OP_LOSS,
    RBP_OP_FUSED,
    RBP_OP_NOTE_USE,
    RBP_OP_LOSS_SEQ,
    RBP_OP_SAMPLE_GATHER,
    RBP_NUM_PHASES,
    RBP_PHASE_DHIDDEN,
    RBP_PHASE_DW,
    RBP_PHASE_LOGITS,
    RBP_PHASE_LOSS,
    RBP_PHASE_MERGE,
    RBP_PHASE_SCALE,
    RBP_PHASE_START,
    RbpError,
    RbpExec,
    alloc_batch,
    lib,
    load_library,
    make_exec,
    make_records,
    make_ring,
    make_sample_cfg,
    policy_logprob_bwd,
    policy_logprob_fwd,
    policy_asymre_fwd_bwd,
    policy_fused_fwd_bwd,
    policy_loss_fwd_bwd,
    policy_loss_seq_fwd_bwd,
    rb_asymre_coef,
    rb_group_advantage,
    rb_hist_accumulate,
    rb_note_use,
    rb_push,
    rb_sample_gather,
    rb_sample_gather_noalloc,
    rbp_workspace_bytes,
    ring_records,
    workspace,
)
