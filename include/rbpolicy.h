/*
 * rbpolicy.h -- C ABI of librbpolicy.so, the MI355X (gfx950) replay-buffer
 * policy-gradient hot path.
 *
 * Method: arXiv 2604.08706, "Efficient RL Training for LLMs with Experience
 * Replay".  A trainer draws stored rollouts from a FIFO replay buffer (Sec. 3.1;
 * App. B "BufferStructure"), re-scores every token under the current policy and
 * trains on it with the clipped, importance-weighted GRPO objective whose old
 * probabilities and group advantages were recorded when the rollout was
 * generated (App. D.2).  This library is that trainer-side path for the LM head:
 *
 *   rb_group_advantage   advantages of a freshly generated group     (App. D.2)
 *   rb_sample_gather     draw records and gather their tokens         (Sec. 3.1, 5; App. B, D.4)
 *   rb_push              append generated groups, FIFO eviction      (App. B, D.2)
 *   rb_note_use          per-record use counts, steps since last use (App. D.3)
 *   rb_hist_accumulate   histograms of the buffer statistics         (Sec. 3.2)
 *   policy_logprob_fwd   log pi(y_t) from hidden states and W         (App. D.2)
 *   policy_loss_fwd_bwd  clipped GRPO loss and d loss / d logp        (App. D.2)
 *   policy_logprob_bwd   d loss / d hidden and d loss / d W           (chain rule of the above)
 *
 * the three token-level calls above in one pass, with the policy entropy:
 *
 *   policy_fused_fwd_bwd forward, loss and backward, 6 d V flop per token (App. D.2, E)
 *
 * and two objective variants on the same tokens:
 *
 *   policy_loss_seq_fwd_bwd  the GRPO objective with the whole-rollout ratio (App. D.2)
 *   rb_asymre_coef,          AsymRE: coefficient at insert and the
 *   policy_asymre_fwd_bwd    objective with its gradient                (App. D.2)
 *
 * Conventions shared by every entry point:
 *   - Pointers marked "device" are HIP device pointers (or managed memory); the
 *     structs themselves and every scalar argument live on the host.
 *   - Tensors are dense, row-major and contiguous.  bf16 tensors are passed as
 *     uint16_t bit patterns (IEEE binary32 truncated to its upper 16 bits).
 *   - The caller owns and allocates every buffer, workspace included; the
 *     library never allocates memory, frees or synchronises.  Size the
 *     workspace with rbp_workspace_bytes().  Workspace contents are scratch
 *     between calls.
 *   - All device work is enqueued on `stream` (a hipStream_t; NULL = the null
 *     stream) and is asynchronous to the host.
 *   - Return value: RBP_OK (0) or a negative RBP_E* code.  Arguments are checked
 *     on the host before anything is enqueued; on an error nothing is enqueued,
 *     except RBP_EHIP, which reports a failed launch (outputs then undefined).
 *     rbp_last_error() gives a thread-local description of the last failure.
 *   - Results are bitwise reproducible for identical inputs (no floating-point
 *     atomics; every reduction runs in a fixed order).
 *   - No exception crosses this interface.  The library holds no mutable global
 *     state except the thread-local error text.
 */
#ifndef RBPOLICY_H
#define RBPOLICY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes --------------------------------------------------------- */
enum {
  RBP_OK = 0,
  RBP_EINVAL = -1,       /* a null pointer, a size out of range, a bad enum     */
  RBP_EUNSUPPORTED = -2, /* a shape the kernels do not handle (e.g. d % 8)      */
  RBP_EWORKSPACE = -3,   /* workspace too small (see rbp_workspace_bytes)       */
  RBP_EHIP = -4          /* a HIP launch failed                                 */
};

/* ---- sampling rules (rb_sample_cfg.mode) ----------------------------------- */
enum {
  RB_UNIFORM = 0,    /* i.i.d. uniform over the live records, with replacement
                        (Sec. 4 analysis; App. C.1)                             */
  RB_POS_MIX = 1,    /* per draw, a coin with probability p_pos picks a uniform
                        positive record (reward > 0), else a uniform live record;
                        no positives -> uniform.  Not in the paper.             */
  RB_POS_RETAIN = 2, /* positive-bias sampling (Sec. 5; App. D.4): uniform over
                        the freshest n_fresh records plus the freshest
                        n_pos_keep positive records older than those            */
  RB_NO_REPLACE = 3, /* uniform without replacement (App. E, "No replacement"):
                        the n_draw slots with the smallest per-slot keys (see
                        rb_sample_cfg), listed in ascending slot order          */
  RB_UNUSED_FIRST = 4 /* without replacement, never-used records first (App. E,
                        "No replacement, at least once"): as RB_NO_REPLACE with
                        records of use_count 0 ranked ahead of used ones        */
};

/* ---- batch layouts (rb_sample_cfg.layout) ---------------------------------- */
enum {
  RB_LAYOUT_PACKED = 0, /* drawn sequences concatenated; one window of the stream */
  RB_LAYOUT_PADDED = 1  /* one row of l_max tokens per draw                        */
};

/* ---- operations for rbp_workspace_bytes ------------------------------------ */
enum {
  RBP_OP_SAMPLE_GATHER = 1, /* n = capacity of the record table              */
  RBP_OP_LOGPROB_FWD = 2,   /* n = T                                          */
  RBP_OP_LOSS = 3,          /* n = T (also policy_asymre_fwd_bwd)            */
  RBP_OP_LOGPROB_BWD = 4,   /* n = tokens per backward chunk (T for one chunk) */
  RBP_OP_LOSS_SEQ = 5,      /* n = B, sequences of policy_loss_seq_fwd_bwd     */
  RBP_OP_FUSED = 6,         /* n = tokens per policy_fused_fwd_bwd chunk       */
  RBP_OP_NOTE_USE = 7       /* n = capacity of the record table              */
};

/*
 * Record table of the replay buffer (App. B "BufferStructure"), as a ring:
 * logical slot s (0 = oldest live record, n_live-1 = newest) is physical row
 * (head + s) % capacity of every per-record array.  A record's tokens and the
 * behaviour log-probabilities recorded at generation (App. D.2) are
 * arena_tokens / arena_old_logp[arena_off .. arena_off + length).
 */
typedef struct rb_records {
  int64_t n_live;                /* live records, 1 <= n_live <= capacity          */
  int64_t capacity;              /* rows of the per-record arrays                  */
  int64_t head;                  /* physical row of slot 0, 0 <= head < capacity   */
  const int64_t* arena_off;      /* device [capacity]                              */
  const int32_t* length;         /* device [capacity], tokens per record (>= 1)    */
  const float* reward;           /* device [capacity]; > 0 means positive/correct  */
  const float* advantage;        /* device [capacity], group advantage at insert   */
  const int32_t* version;        /* device [capacity], policy version at generation*/
  const int32_t* arena_tokens;   /* device [arena_size]                            */
  const float* arena_old_logp;   /* device [arena_size]                            */
  int64_t arena_size;            /* every record must lie inside [0, arena_size)   */
  const int32_t* use_count;      /* device [capacity], samples per row so far
                                    (rb_note_use); read by RB_UNUSED_FIRST only,
                                    may be NULL for the other modes               */
} rb_records;

/*
 * Sampling configuration.  Draw j of a call reads the Philox4x64-10 block with
 * counter (j, step, 0, 0) and key (seed, 0) (Salmon et al., SC'11); its first
 * word x0 maps to an index in [0, n) as floor(x0 * n / 2^64), the high half of
 * its second word x1 decides the stratum coin: (x1 >> 32) < p_pos_q32.  A call
 * therefore depends only on (seed, step) and the record table: re-running a
 * step after a restart reproduces it bit for bit.  The modes without
 * replacement give slot s the key x0 >> 1 of the block with counter
 * (s, step, 1, 0) and the same key (RB_UNUSED_FIRST adds 2^63 when the slot's
 * use_count is > 0) and take the n_draw smallest (key, slot) pairs.
 */
typedef struct rb_sample_cfg {
  int32_t mode;          /* RB_UNIFORM, RB_POS_MIX, RB_POS_RETAIN, RB_NO_REPLACE,
                            RB_UNUSED_FIRST                                        */
  int32_t layout;        /* RB_LAYOUT_PACKED / RB_LAYOUT_PADDED                    */
  uint64_t seed;
  uint64_t step;
  int64_t n_draw;        /* draws (sequences) in the batch, 1 .. 2^20              */
  uint64_t p_pos_q32;    /* RB_POS_MIX: floor(p_pos * 2^32), 0 .. 2^32             */
  int64_t n_fresh;       /* RB_POS_RETAIN: (1 - delta) N                           */
  int64_t n_pos_keep;    /* RB_POS_RETAIN: floor(delta N)                          */
  int32_t cur_version;   /* current policy version; age = cur_version - version    */
  int32_t pad_;
  int64_t max_tokens;    /* packed: window length (token capacity of the outputs)  */
  int64_t token_begin;   /* packed: window start within the concatenated stream   */
  int64_t l_max;         /* padded: row length                                     */
} rb_sample_cfg;

/*
 * Outputs of rb_sample_gather, all caller-allocated device buffers.
 * Packed: tokens / old_logp / seq_of_token have max_tokens entries; position t
 *   holds stream position token_begin + t; past the end of the stream the
 *   padding is token 0, old_logp 0, seq_of_token -1.  cu_seqlens[j] is the
 *   stream position where draw j starts (prefix sums of full lengths).
 * Padded: those arrays are [n_draw, l_max]; row j holds the first
 *   min(len_j, l_max) tokens of draw j, then padding; cu_seqlens[j] = j * l_max.
 * Per draw j: idx = slot drawn, adv = its advantage, len = its full length,
 *   age = cur_version - its version.  n_tokens = valid output positions.
 */
typedef struct rb_batch {
  int32_t* idx;          /* device [n_draw]                                        */
  float* adv;            /* device [n_draw]                                        */
  int32_t* len;          /* device [n_draw]                                        */
  int32_t* age;          /* device [n_draw]                                        */
  int32_t* cu_seqlens;   /* device [n_draw + 1]                                    */
  int32_t* tokens;       /* device, see above                                      */
  float* old_logp;       /* device, see above                                      */
  int32_t* seq_of_token; /* device, see above; -1 marks padding                    */
  int64_t* n_tokens;     /* device [1]                                             */
} rb_batch;

/*
 * Draw a training batch from the replay buffer and gather it (Sec. 3.1:
 * sampling does not remove records; Sec. 4: draws are uniform with
 * replacement; Sec. 5 and App. D.4: positive-bias retention; App. E: the
 * variants without replacement).  Draws are kept in draw order, duplicates
 * included; the modes without replacement list distinct slots ascending.
 * Errors: RBP_EINVAL for null pointers, n_live outside [1, capacity], n_draw
 *   outside [1, 2^20] (or above n_live without replacement), a null
 *   use_count for RB_UNUSED_FIRST, an unknown mode/layout, p_pos_q32 > 2^32, negative
 *   n_fresh/n_pos_keep, max_tokens < 1 (packed) or l_max < 1 (padded);
 *   RBP_EWORKSPACE if ws_bytes < rbp_workspace_bytes(RBP_OP_SAMPLE_GATHER,
 *   capacity, 0, 0).  Record offsets and lengths are trusted: the caller
 *   guarantees each record lies inside the arena and the stream fits in
 *   int32 positions.  RB_POS_RETAIN with an empty retained set draws slot 0.
 */
int rb_sample_gather(const rb_records* rec, const rb_sample_cfg* cfg,
                     const rb_batch* out, void* ws, size_t ws_bytes,
                     void* stream);

/*
 * rb_sample_gather without a workspace argument, for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same arguments (minus ws, ws_bytes), same results bit
 * for bit, same errors.  Its workspace is a static device array of 32 MiB
 * that each GPU the library runs on holds from module load until the
 * process ends; the call allocates and frees nothing.  Record tables whose
 * rbp_workspace_bytes(RBP_OP_SAMPLE_GATHER, capacity, 0, 0) exceeds 32 MiB
 * (capacity above about 1.6 million records) are rejected with
 * RBP_EWORKSPACE before anything is enqueued.  Every call on a GPU uses that
 * GPU's one array: calls that may overlap on the same GPU (two streams, two
 * threads) race and must be ordered by the caller.  The first call on a
 * device resolves the array's device address (hipGetSymbolAddress) and
 * should run outside graph capture.
 */
int rb_sample_gather_noalloc(const rb_records* rec, const rb_sample_cfg* cfg,
                             const rb_batch* out, void* stream);

/*
 * Group-normalised advantage at insert time (App. D.2):
 * A_i = (r_i - mean_g) / (std_g + eps) over group g = [group_off[g],
 * group_off[g+1]); std uses `ddof` (1 = sample estimate); a group whose rewards
 * are all equal (or has no degrees of freedom) gets A = 0 exactly.  The
 * mean, std and quotient are formed in fp64 (fp32 inputs sum exactly there),
 * then A is rounded to fp32.  reward, group_off, adv: device fp32 / int32.  Groups must be non-overlapping, ascending.
 * Errors: RBP_EINVAL for null pointers, n_groups < 0, ddof not 0 or 1, eps < 0.
 */
int rb_group_advantage(const float* reward, const int32_t* group_off,
                       int32_t n_groups, int32_t ddof, float eps, float* adv,
                       void* stream);

/*
 * Per-token log-probability of the sampled tokens under the current policy
 * (App. D.2, temperature 1): z_t = W h_t, lse_t = log sum_v exp(z_{t,v}),
 * logp_t = z_{t,y_t} - lse_t.  bf16 MFMA products with fp32 accumulation; the
 * T x V logits are never written to memory (online log-sum-exp per tile).
 * hidden  device bf16 [T, d];  W device bf16 [V, d];  tokens device int32 [T]
 *         (each in [0, V) where not masked);
 * seq_of_token device int32 [T] or NULL; a negative entry masks the token
 *         (logp = 0, lse = 0);
 * logp, lse device fp32 [T] (lse is what policy_logprob_bwd needs);
 * ws      device, >= rbp_workspace_bytes(RBP_OP_LOGPROB_FWD, T, d, V).
 * Errors: RBP_EINVAL (null pointers, T < 0, d < 1, V < 1);
 *         RBP_EUNSUPPORTED (d % 8 != 0); RBP_EWORKSPACE.
 */
int policy_logprob_fwd(const uint16_t* hidden, const uint16_t* W,
                       const int32_t* tokens, const int32_t* seq_of_token,
                       int64_t T, int32_t d, int32_t V, float* logp, float* lse,
                       void* ws, size_t ws_bytes, void* stream);

/*
 * Clipped, importance-weighted GRPO objective on replayed tokens and its
 * gradient (App. D.2), token-level ratio with per-sequence token means:
 *   rho_t   = exp(logp_t - old_logp_t)
 *   l_t     = min(rho_t A_i, clip(rho_t, 1 - eps_low, 1 + eps_high) A_i)
 *   loss    = -sum_t l_t / (n_seq_total * seq_len_i)      (i = seq_of_token[t])
 *   dlogp_t = -A_i rho_t act_t / (n_seq_total * seq_len_i), act_t = 0 iff
 *             (A_i > 0 and rho_t > 1 + eps_high) or (A_i < 0 and rho_t < 1 - eps_low).
 * logp, old_logp, seq_of_token device [T]; adv device fp32 [B]; seq_len device
 * int32 [B] (full lengths, >= 1); tokens with seq_of_token < 0 are masked
 * (dlogp = 0).  seq_of_token entries must be < B.
 * loss_accum device fp32 [1] and stats device fp32 [4] are ACCUMULATED (+=):
 *   stats = {sum rho, tokens clipped with zero gradient, valid tokens, sum l_t}.
 * dlogp device fp32 [T] is overwritten.
 * ws device, >= rbp_workspace_bytes(RBP_OP_LOSS, T, 0, 0).
 * Errors: RBP_EINVAL (null pointers, T < 0, B < 1, n_seq_total < 1, eps < 0);
 *         RBP_EWORKSPACE.
 */
int policy_loss_fwd_bwd(const float* logp, const float* old_logp,
                        const int32_t* seq_of_token, const float* adv,
                        const int32_t* seq_len, int64_t T, int32_t B,
                        int64_t n_seq_total, float eps_low, float eps_high,
                        float* loss_accum, float* dlogp, float* stats,
                        void* ws, size_t ws_bytes, void* stream);

/*
 * Whole-sequence-ratio form of the same objective -- the printed App. D.2
 * formula read literally (the ratio of the rollout's probabilities):
 *   rho_i   = exp(sum_{t in i} (logp_t - old_logp_t))
 *   l_i     = min(rho_i A_i, clip(rho_i, 1 - eps_low, 1 + eps_high) A_i)
 *   loss    = -sum_i l_i / n_seq_total
 *   dlogp_t = -A_i rho_i act_i / n_seq_total for every token t of sequence i,
 *             act_i as above with rho_i.
 * Sequence i is tokens [cu_seqlens[i], cu_seqlens[i+1]) and must be complete
 * in this call (the ratio needs every token); tokens from cu_seqlens[B] to T
 * get dlogp = 0.  logp, old_logp device fp32 [T]; cu_seqlens device int32
 * [B + 1], non-decreasing, cu_seqlens[0] = 0, cu_seqlens[B] <= T; adv device
 * fp32 [B].  loss_accum [1] and stats [4] ACCUMULATE:
 *   stats = {sum rho_i, sequences clipped with zero gradient, sequences, sum l_i}.
 * ws device, >= rbp_workspace_bytes(RBP_OP_LOSS_SEQ, B, 0, 0).
 * Errors: RBP_EINVAL (null pointers, T < 0, B < 1, n_seq_total < 1, eps < 0);
 *         RBP_EWORKSPACE.
 */
int policy_loss_seq_fwd_bwd(const float* logp, const float* old_logp,
                            const int32_t* cu_seqlens, const float* adv, int64_t T,
                            int32_t B, int64_t n_seq_total, float eps_low, float eps_high,
                            float* loss_accum, float* dlogp, float* stats, void* ws,
                            size_t ws_bytes, void* stream);

/*
 * AsymRE coefficient at insert (App. D.2): for every record of group g
 * (records [group_off[g], group_off[g+1])),
 *   coef_i = reward_i - (mean reward of the group + delta_v),
 * the paper's delta_v being -0.1.  Stored in the record table's advantage
 * slot when training with policy_asymre_fwd_bwd.  Formed in fp64, rounded
 * to fp32 once.  reward, coef device fp32;
 * group_off device int32 [n_groups + 1].
 * Errors: RBP_EINVAL (null pointers, n_groups < 0).
 */
int rb_asymre_coef(const float* reward, const int32_t* group_off, int32_t n_groups,
                   float delta_v, float* coef, void* stream);

/*
 * AsymRE objective (App. D.2) on replayed tokens, no ratio and no clip:
 *   loss    = -sum_t coef_i logp_t / n_seq_total       (i = seq_of_token[t])
 *   dlogp_t = -coef_i / n_seq_total
 * logp, seq_of_token device [T] (seq_of_token < 0 masks the token: dlogp = 0);
 * coef device fp32 [B] (rb_asymre_coef).  loss_accum [1] and stats [2]
 * ACCUMULATE: stats = {valid tokens, sum coef_i logp_t}.  dlogp overwritten.
 * ws device, >= rbp_workspace_bytes(RBP_OP_LOSS, T, 0, 0).
 * Errors: RBP_EINVAL (null pointers, T < 0, B < 1, n_seq_total < 1);
 *         RBP_EWORKSPACE.
 */
int policy_asymre_fwd_bwd(const float* logp, const int32_t* seq_of_token, const float* coef,
                          int64_t T, int32_t B, int64_t n_seq_total, float* loss_accum,
                          float* dlogp, float* stats, void* ws, size_t ws_bytes,
                          void* stream);

/*
 * Backward of policy_logprob_fwd: with p_t = exp(z_t - lse_t) and
 * dz_t = dlogp_t (e_{y_t} - p_t):  dhidden_t = W^T dz_t,  dW (+)= sum_t dz_t h_t^T.
 * The logits are recomputed tile by tile (bf16 MFMA, fp32 accumulation); dz is
 * rounded to bf16 for the two products.  Masked tokens get a zero dhidden row
 * and add nothing to dW.
 * hidden, W, tokens, seq_of_token as in policy_logprob_fwd; lse, dlogp device
 * fp32 [T]; dhidden device fp32 [T, d] (overwritten); dW device fp32 [V, d]
 * (overwritten, or accumulated into when accumulate_dW != 0).
 * ws device: the tokens are processed in chunks of Tc tokens, with Tc the
 * largest multiple of 256 (at most T rounded up to 256) whose
 * rbp_workspace_bytes(RBP_OP_LOGPROB_BWD, Tc, d, V) fits in ws_bytes.  With
 * Vp = V rounded up to 256 it holds dz^T (bf16 [Vp, Tc]) and a split-K
 * partial of dhidden (fp32 [Tc, d]): 5.2 GB for Tc = 16384 at d = 3584,
 * V = 152064.
 * Errors: RBP_EINVAL; RBP_EUNSUPPORTED (d % 8 != 0); RBP_EWORKSPACE (not even
 * a 256-token chunk fits).
 */
int policy_logprob_bwd(const uint16_t* hidden, const uint16_t* W,
                       const int32_t* tokens, const int32_t* seq_of_token,
                       const float* lse, const float* dlogp, int64_t T,
                       int32_t d, int32_t V, float* dhidden, float* dW,
                       int accumulate_dW, void* ws, size_t ws_bytes,
                       void* stream);

/*
 * Optional phase events of policy_fused_fwd_bwd, owned by the caller (the
 * library keeps nothing between calls): phase_event[k], a hipEvent_t or
 * NULL, is recorded on `stream` when phase k of a chunk is done
 * (RBP_PHASE_*), for timing the phases without a profiler; with several
 * chunks a later record replaces an earlier one.  Leave them NULL under
 * graph capture.
 */
enum {
  RBP_PHASE_START = 0,    /* before the chunk's first kernel                    */
  RBP_PHASE_LOGITS = 1,   /* target logits and the logit tile pass done         */
  RBP_PHASE_MERGE = 2,    /* lse, logp and entropy done                         */
  RBP_PHASE_LOSS = 3,     /* loss pass done (dlogp)                             */
  RBP_PHASE_SCALE = 4,    /* per-token scales, scaled hidden states done        */
  RBP_PHASE_DW = 5,       /* dW done                                            */
  RBP_PHASE_DHIDDEN = 6,  /* dhidden done                                       */
  RBP_NUM_PHASES = 7
};

typedef struct rbp_exec {
  void* phase_event[RBP_NUM_PHASES];  /* hipEvent_t or NULL each                */
} rbp_exec;

/*
 * policy_logprob_fwd + policy_loss_fwd_bwd + policy_logprob_bwd in one pass,
 * plus the per-token entropy of the policy, H_t = -sum_v p_{t,v} log p_{t,v}
 * (the training entropy of App. E).  The separate calls execute 8 d V flop
 * per token because the backward recomputes the logits; this one executes the
 * 6 d V of the definition by keeping, per token and vocabulary entry, the
 * forward tile pass's exponential exp(z - R_t) as bf16 in the workspace (2 V
 * bytes per token: a T x V array, which policy_logprob_fwd never holds).  The
 * per-token reference R_t = z_{t,y_t} - old_logp_t is the log-sum-exp the
 * behaviour log-prob implies (lse_t - log rho_t), so the stored values are
 * p_{t,v} / rho_t and the backward's dz is one scalar per token times them:
 * the logits never reach memory and no pass over the array rescales it.
 * A token whose R_t lies too far from its logits for exp(z - R_t) to stay in
 * range -- R_t below M_t - 20 or above M_t + 40 to 47 (M_t its largest
 * logit: a ratio below about e^-20 or above about e^40), or an invalid
 * old_logp -- is re-referenced to its largest logit by a pass over its
 * column alone.  dz is rounded to
 * bf16 once (as exp(z - R_t)); the dW product reads h_t scaled by the token's
 * factor, rounded to bf16.
 * exec: NULL, or the caller's rbp_exec of phase events.
 * Arguments: hidden, W, tokens, seq_of_token as in policy_logprob_fwd
 * (seq_of_token required); old_logp, adv, seq_len, B, n_seq_total, eps_low,
 * eps_high, loss_accum, stats as in policy_loss_fwd_bwd (loss_accum and stats
 * ACCUMULATE); logp, lse, dlogp device fp32 [T] (overwritten); entropy device
 * fp32 [T] (overwritten; may be NULL; 0 for masked tokens); dhidden, dW,
 * accumulate_dW as in policy_logprob_bwd.
 * ws device: tokens are processed in chunks of Tc tokens, with Tc the largest
 * multiple of 256 (at most T rounded up to 256, at most 2^21) whose
 * rbp_workspace_bytes(RBP_OP_FUSED, Tc, d, V) fits in ws_bytes: with
 * Vp = V rounded up to 256, bf16 [Vp, Tc], fp32 [3 Vp / 128, Tc] partial
 * sums, five fp32 / int32 [Tc] arrays, bf16 [Tc, d] (scaled hidden states),
 * fp32 [Tc, d] and the loss pass's sums -- 5.6 GB for Tc = 16384 at
 * d = 3584, V = 152064.
 * Errors: RBP_EINVAL (null pointers, T < 0, d < 1, V < 1, B < 1,
 *         n_seq_total < 1, eps < 0); RBP_EUNSUPPORTED (d % 8 != 0);
 *         RBP_EWORKSPACE (not even a 256-token chunk fits); RBP_EHIP (a
 *         launch or a phase-event record failed: earlier work may still be
 *         pending on `stream`).
 */
int policy_fused_fwd_bwd(const uint16_t* hidden, const uint16_t* W,
                         const int32_t* tokens, const int32_t* seq_of_token,
                         const float* old_logp, const float* adv,
                         const int32_t* seq_len, int64_t T, int32_t d, int32_t V,
                         int32_t B, int64_t n_seq_total, float eps_low,
                         float eps_high, float* logp, float* lse, float* entropy,
                         float* loss_accum, float* dlogp, float* stats,
                         float* dhidden, float* dW, int accumulate_dW, void* ws,
                         size_t ws_bytes, const rbp_exec* exec, void* stream);

/*
 * The record table as rb_push writes it: the rb_records arrays, writable, with
 * a fixed arena stretch of slot_tokens tokens per row (row r owns
 * arena[r * slot_tokens, (r + 1) * slot_tokens)), so that a new record always
 * reuses the storage of the record it evicts.
 */
typedef struct rb_ring {
  int64_t n_live;            /* host; updated by rb_push                           */
  int64_t capacity;          /* N, rows of every per-record array                  */
  int64_t head;              /* host; physical row of slot 0, updated by rb_push   */
  int64_t slot_tokens;       /* arena tokens per row (>= 1)                        */
  int64_t* arena_off;        /* device [capacity]                                  */
  int32_t* length;           /* device [capacity]                                  */
  float* reward;             /* device [capacity]                                  */
  float* advantage;          /* device [capacity]                                  */
  int32_t* version;          /* device [capacity]                                  */
  int32_t* use_count;        /* device [capacity] or NULL: reset to 0 on insert     */
  int64_t* last_step;        /* device [capacity] or NULL: reset to -1 on insert    */
  int32_t* arena_tokens;     /* device [capacity * slot_tokens]                    */
  float* arena_old_logp;     /* device [capacity * slot_tokens]                    */
  int64_t* replay_hist;      /* device [replay_bins] or NULL: replay ratios of the
                                records a push evicts, added to (see rb_push)     */
  int32_t replay_bins;       /* 1 .. 4096 when replay_hist is set                  */
  int32_t pad_;
} rb_ring;

/*
 * Append freshly generated groups to the buffer, first in first out (App. B
 * "BufferStructure": a push into a full buffer evicts the oldest record), and
 * record each rollout's group advantage as rb_group_advantage computes it
 * (App. D.2: advantages are fixed at generation).  New record i (0-based, in
 * the given order) goes to physical row (head + n_live + i) % capacity; then
 * n_live = min(capacity, n_live + n_new) and head moves past the evicted rows.
 * group_off device int32 [n_groups + 1] splits the n_new records into groups
 * (group_off[0] = 0, group_off[n_groups] = n_new); length (each >= 1),
 * reward device [n_new]; src_off device int64 [n_new]: record i's tokens / behaviour
 * log-probs are tokens / old_logp[src_off[i] .. + length[i]).  A record longer
 * than slot_tokens keeps its first slot_tokens tokens (its stored length is
 * cut to that).  version is stored for every new record.  The device-side
 * group_off, length and src_off are trusted (not read on the host): offsets
 * outside the given arrays are the caller's error.
 * Replay ratios (Sec. 3.2: the number of gradient steps that used a
 * rollout): when replay_hist is set, each evicted record's final use_count u
 * adds 1 to replay_hist[min(u, replay_bins - 1)] before its row is reused
 * (needs use_count; integer atomics, order-free).
 * Errors: RBP_EINVAL (null pointers, n_new outside [1, capacity],
 *         n_groups < 1, n_live outside [0, capacity], head outside
 *         [0, capacity), slot_tokens < 1, ddof not 0 or 1, eps < 0,
 *         replay_hist without use_count or with replay_bins outside
 *         [1, 4096]).
 */
int rb_push(rb_ring* ring, int32_t n_new, int32_t n_groups, const int32_t* group_off,
            const int32_t* length, const int64_t* src_off, const float* reward,
            int32_t version, const int32_t* tokens, const float* old_logp,
            int32_t ddof, float eps, void* stream);

/*
 * Usage bookkeeping after a batch is drawn (App. D.3, "Steps-since-last-use"):
 * for draw j in draw order, since[j] = -1 if its record was never used before
 * ("new"), 0 if an earlier draw of this batch took the same record, else
 * step - last_step of the record; then every drawn record gets
 * last_step = step and use_count += its number of draws.  idx device int32
 * [n_draw] (slots as rb_sample_gather writes them, trusted to lie below the
 * table's n_live); head, capacity as in the record table; use_count device int32, last_step device int64 [capacity];
 * since device int32 [n_draw] (may be NULL).  Steps must not decrease
 * between calls.
 * ws device, >= rbp_workspace_bytes(RBP_OP_NOTE_USE, capacity, 0, 0).
 * Errors: RBP_EINVAL (null pointers, n_draw < 0, head outside [0, capacity),
 *         step < 0); RBP_EWORKSPACE.
 */
int rb_note_use(const int32_t* idx, int64_t n_draw, int64_t head, int64_t capacity,
                int64_t step, int32_t* use_count, int64_t* last_step, int32_t* since,
                void* ws, size_t ws_bytes, void* stream);

/*
 * Buffer statistics as histograms (Sec. 3.2: the distributions of
 * off-policiness, replay ratio and steps since last use): value v of
 * values device int32 [n] adds 1 to hist[min(max(v - lo, 0), n_bins - 1)].
 * Typical inputs: the age output of rb_sample_gather (off-policiness, lo =
 * 0), the since output of rb_note_use (lo = -1, so "new" has bin 0), a
 * use_count array (replay ratios of live records, lo = 0).  hist device
 * int64 [n_bins], ADDED to; integer atomics, so the counts do not depend on
 * the order of the additions.
 * Errors: RBP_EINVAL (n < 0, n_bins outside [1, 4096], null pointers when
 *         n > 0).
 */
int rb_hist_accumulate(const int32_t* values, int64_t n, int32_t lo, int32_t n_bins,
                       int64_t* hist, void* stream);

/* Workspace bytes an operation needs (see RBP_OP_*); 0 for an invalid op. */
size_t rbp_workspace_bytes(int op, int64_t n, int32_t d, int32_t V);

/* Static text for a status code. */
const char* rbp_status_string(int status);

/* Thread-local description of the last failure in this thread ("" if none). */
const char* rbp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* RBPOLICY_H */
