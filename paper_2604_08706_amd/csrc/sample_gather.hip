// Replay-buffer sampling and batch gather (rb_sample_gather).
//
// Paper: the buffer is a FIFO list whose sampling does not remove records
// (Sec. 3.1; App. B "BufferStructure"); draws are uniform with replacement
// (Sec. 4); positive-bias retention keeps the freshest (1-delta)N rollouts
// plus the freshest delta*N correct rollouts older than those (Sec. 5;
// App. D.4).  The positive-prioritised mixture is an addition (see header).
//
// Device pipeline (one stream):
//   [mix/retain only] pos_count -> pos_scan -> pos_compact : ascending list of
//       positive slots (slot = FIFO position, 0 = oldest) in the workspace;
//   [without replacement] slot_key -> 8 x (select_hist -> select_digit) ->
//       sel_count -> sel_scan -> sel_compact : an MSD radix select finds the
//       n_draw-th smallest 64-bit slot key K exactly, then the slots with a key
//       below K (and the first ties in slot order) are listed ascending;
//   draw     : one thread per draw; Philox4x64-10 block -> slot; per-draw
//              outputs; block scan of lengths -> cu_seqlens, n_tokens;
//   gather   : one thread per output position; coalesced copies from the
//              token arena.
// Everything is integer work or a bit-exact copy of stored floats.

#include "rbp_internal.h"

namespace {

constexpr int kSlotsPerBlock = 1024;  // compaction granule
constexpr int kCountThreads = 256;    // 4 slots per thread
constexpr int kDrawThreads = 1024;

// ---- Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11) ----------------------
struct Block4 {
  uint64_t x0, x1, x2, x3;
};

__device__ __forceinline__ Block4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2,
                                                uint64_t c3, uint64_t k0, uint64_t k1) {
  const uint64_t kMul0 = 0xD2E7470EE14C6C93ull, kMul1 = 0xCA5A826395121157ull;
  const uint64_t kWeyl0 = 0x9E3779B97F4A7C15ull, kWeyl1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += kWeyl0;
      k1 += kWeyl1;
    }
    const uint64_t hi0 = __umul64hi(kMul0, c0), lo0 = kMul0 * c0;
    const uint64_t hi1 = __umul64hi(kMul1, c2), lo1 = kMul1 * c2;
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return {c0, c1, c2, c3};
}

__device__ __forceinline__ int64_t phys_row(int64_t slot, int64_t head, int64_t cap) {
  int64_t r = head + slot;
  return r >= cap ? r - cap : r;
}

// Block-wide exclusive scan of one int64 per thread (fixed order).
template <int NT>
__device__ int64_t block_exclusive_scan(int64_t v, int64_t* total, int64_t* lds_waves) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int64_t incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int64_t o = __shfl_up(incl, off, 64);
    if (lane >= off) incl += o;
  }
  if (lane == 63) lds_waves[wave] = incl;
  __syncthreads();
  int64_t wave_base = 0, sum = 0;
  for (int w = 0; w < NT / 64; ++w) {
    if (w < wave) wave_base += lds_waves[w];
    sum += lds_waves[w];
  }
  __syncthreads();
  *total = sum;
  return wave_base + incl - v;
}

__global__ void __launch_bounds__(kCountThreads) pos_count_kernel(
    const float* __restrict__ reward, int64_t head, int64_t cap, int64_t n_range,
    int32_t* __restrict__ counts) {
  __shared__ int64_t lds[kCountThreads / 64];
  const int64_t s0 = (int64_t)blockIdx.x * kSlotsPerBlock + threadIdx.x * 4;
  int64_t c = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t s = s0 + i;
    if (s < n_range && reward[phys_row(s, head, cap)] > 0.0f) ++c;
  }
  int64_t total;
  block_exclusive_scan<kCountThreads>(c, &total, lds);
  if (threadIdx.x == 0) counts[blockIdx.x] = (int32_t)total;
}

__global__ void __launch_bounds__(1024) pos_scan_kernel(const int32_t* __restrict__ counts,
                                                        int32_t* __restrict__ offsets,
                                                        int64_t nb, int64_t* __restrict__ meta) {
  __shared__ int64_t lds[1024 / 64];
  int64_t carry = 0;
  for (int64_t base = 0; base < nb; base += 1024) {
    const int64_t i = base + threadIdx.x;
    const int64_t v = i < nb ? counts[i] : 0;
    int64_t total;
    const int64_t ex = block_exclusive_scan<1024>(v, &total, lds);
    if (i < nb) offsets[i] = (int32_t)(carry + ex);
    carry += total;
  }
  if (threadIdx.x == 0) meta[0] = carry;
}

__global__ void __launch_bounds__(kCountThreads) pos_compact_kernel(
    const float* __restrict__ reward, int64_t head, int64_t cap, int64_t n_range,
    const int32_t* __restrict__ offsets, int32_t* __restrict__ pos_list) {
  __shared__ int64_t lds[kCountThreads / 64];
  const int64_t s0 = (int64_t)blockIdx.x * kSlotsPerBlock + threadIdx.x * 4;
  bool f[4];
  int64_t c = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t s = s0 + i;
    f[i] = s < n_range && reward[phys_row(s, head, cap)] > 0.0f;
    c += f[i];
  }
  int64_t total;
  int64_t at = offsets[blockIdx.x] + block_exclusive_scan<kCountThreads>(c, &total, lds);
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (f[i]) pos_list[at++] = (int32_t)(s0 + i);
}

// ---- selection without replacement -----------------------------------------

// Key of slot s: the top 63 bits of word 0 of the Philox block with counter
// (s, step, 1, 0); for never-used-first, bit 63 set when the slot was used.
__global__ void __launch_bounds__(256) slot_key_kernel(uint64_t seed, uint64_t step,
                                                       int64_t n_live, int64_t head, int64_t cap,
                                                       const int32_t* __restrict__ use_count,
                                                       uint64_t* __restrict__ keys) {
  for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < n_live;
       s += (int64_t)gridDim.x * 256) {
    uint64_t k = philox4x64_10((uint64_t)s, step, 1, 0, seed, 0).x0 >> 1;
    if (use_count != nullptr && use_count[phys_row(s, head, cap)] > 0) k |= 1ull << 63;
    keys[s] = k;
  }
}

// Radix-select state: the key digits fixed so far, how many keys still to be
// taken among those sharing them, and the histogram of the next digit.
struct SelState {
  uint64_t prefix;
  int64_t need;
  uint32_t hist[256];
};

__global__ void __launch_bounds__(256) select_init_kernel(SelState* st, int64_t n_draw) {
  st->hist[threadIdx.x] = 0u;
  if (threadIdx.x == 0) {
    st->prefix = 0;
    st->need = n_draw;
  }
}

// Histogram of digit `pass` (bits 56 - 8 pass .. +8, most significant first)
// over the keys whose higher digits equal the prefix.  Integer atomics: the
// counts do not depend on the order of the additions.
__global__ void __launch_bounds__(256) select_hist_kernel(const uint64_t* __restrict__ keys,
                                                          int64_t n, int pass,
                                                          SelState* __restrict__ st) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0u;
  __syncthreads();
  const int shift = 56 - 8 * pass;
  const uint64_t hi = pass == 0 ? 0 : st->prefix >> (shift + 8);
  for (int64_t s = (int64_t)blockIdx.x * 256 + threadIdx.x; s < n;
       s += (int64_t)gridDim.x * 256) {
    const uint64_t k = keys[s];
    if (pass == 0 || (k >> (shift + 8)) == hi) atomicAdd(&h[(k >> shift) & 255u], 1u);
  }
  __syncthreads();
  if (h[threadIdx.x] != 0u) atomicAdd(&st->hist[threadIdx.x], h[threadIdx.x]);
}

// The digit holding the need-th smallest remaining key; clears the histogram.
__global__ void __launch_bounds__(256) select_digit_kernel(int pass, SelState* __restrict__ st) {
  if (threadIdx.x == 0) {
    int64_t cum = 0;
    int d = 0;
    for (; d < 255; ++d) {
      if (cum + (int64_t)st->hist[d] >= st->need) break;
      cum += st->hist[d];
    }
    st->need -= cum;
    st->prefix |= (uint64_t)d << (56 - 8 * pass);
  }
  __syncthreads();
  st->hist[threadIdx.x] = 0u;
}

// Per slot, (key < K) in the low 32 bits and (key == K) in the high 32 bits:
// one int64 whose block sums carry both counts.
__device__ __forceinline__ int64_t sel_flags(uint64_t k, uint64_t K) {
  return (k < K ? 1 : 0) + (k == K ? (int64_t(1) << 32) : 0);
}

__global__ void __launch_bounds__(kCountThreads) sel_count_kernel(
    const uint64_t* __restrict__ keys, int64_t n, const SelState* __restrict__ st,
    int64_t* __restrict__ counts) {
  __shared__ int64_t lds[kCountThreads / 64];
  const uint64_t K = st->prefix;
  const int64_t s0 = (int64_t)blockIdx.x * kSlotsPerBlock + threadIdx.x * 4;
  int64_t c = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i)
    if (s0 + i < n) c += sel_flags(keys[s0 + i], K);
  int64_t total;
  block_exclusive_scan<kCountThreads>(c, &total, lds);
  if (threadIdx.x == 0) counts[blockIdx.x] = total;
}

__global__ void __launch_bounds__(1024) sel_scan_kernel(const int64_t* __restrict__ counts,
                                                        int64_t* __restrict__ offsets,
                                                        int64_t nb) {
  __shared__ int64_t lds[1024 / 64];
  int64_t carry = 0;
  for (int64_t base = 0; base < nb; base += 1024) {
    const int64_t i = base + threadIdx.x;
    const int64_t v = i < nb ? counts[i] : 0;
    int64_t total;
    const int64_t ex = block_exclusive_scan<1024>(v, &total, lds);
    if (i < nb) offsets[i] = carry + ex;
    carry += total;
  }
}

// A slot with key < K goes to position (# keys < K before it) + min(# ties
// before it, need); a tie is taken while fewer than `need` ties precede it.
__global__ void __launch_bounds__(kCountThreads) sel_compact_kernel(
    const uint64_t* __restrict__ keys, int64_t n, const SelState* __restrict__ st,
    const int64_t* __restrict__ offsets, int32_t* __restrict__ sel) {
  __shared__ int64_t lds[kCountThreads / 64];
  const uint64_t K = st->prefix;
  const int64_t need = st->need;
  const int64_t s0 = (int64_t)blockIdx.x * kSlotsPerBlock + threadIdx.x * 4;
  int64_t f[4], c = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[i] = s0 + i < n ? sel_flags(keys[s0 + i], K) : 0;
    c += f[i];
  }
  int64_t total;
  int64_t at = offsets[blockIdx.x] + block_exclusive_scan<kCountThreads>(c, &total, lds);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t less = at & 0xffffffffll, ties = at >> 32;
    if (f[i] == 1)
      sel[less + (ties < need ? ties : need)] = (int32_t)(s0 + i);
    else if (f[i] != 0 && ties < need)
      sel[less + ties] = (int32_t)(s0 + i);
    at += f[i];
  }
}

struct DrawParams {
  int32_t mode, layout;
  uint64_t seed, step, p_q32;
  int64_t n_draw, n_live, head, cap;
  int64_t first_fresh, n_pos_keep;
  int32_t cur_version;
  int64_t max_tokens, token_begin, l_max;
};

__global__ void __launch_bounds__(kDrawThreads) draw_kernel(
    DrawParams p, const int64_t* __restrict__ meta, const int32_t* __restrict__ pos_list,
    const int32_t* __restrict__ length, const float* __restrict__ advantage,
    const int32_t* __restrict__ version, int32_t* __restrict__ out_idx,
    float* __restrict__ out_adv, int32_t* __restrict__ out_len, int32_t* __restrict__ out_age,
    int32_t* __restrict__ cu_seqlens, int64_t* __restrict__ n_tokens,
    int64_t* __restrict__ stream_total) {
  __shared__ int64_t lds[kDrawThreads / 64];
  const int64_t n_pos = (p.mode == RB_POS_MIX || p.mode == RB_POS_RETAIN) ? meta[0] : 0;
  // retained set: the newest `keep` positives older than the fresh part, then
  // the fresh part [first_fresh, n_live)
  const int64_t keep = n_pos < p.n_pos_keep ? n_pos : p.n_pos_keep;
  const int64_t n_set = keep + (p.n_live - p.first_fresh);
  int64_t carry = 0, valid = 0;
  if (threadIdx.x == 0) cu_seqlens[0] = 0;
  for (int64_t base = 0; base < p.n_draw; base += kDrawThreads) {
    const int64_t j = base + threadIdx.x;
    int64_t len = 0;
    if (j < p.n_draw) {
      const Block4 b = philox4x64_10((uint64_t)j, p.step, 0, 0, p.seed, 0);
      int64_t slot;
      if (p.mode == RB_UNIFORM) {
        slot = (int64_t)__umul64hi(b.x0, (uint64_t)p.n_live);
      } else if (p.mode == RB_POS_MIX) {
        if (n_pos > 0 && (b.x1 >> 32) < p.p_q32)
          slot = pos_list[__umul64hi(b.x0, (uint64_t)n_pos)];
        else
          slot = (int64_t)__umul64hi(b.x0, (uint64_t)p.n_live);
      } else if (p.mode == RB_NO_REPLACE || p.mode == RB_UNUSED_FIRST) {
        slot = pos_list[j];  // the selected slots, ascending
      } else {
        if (n_set <= 0) {
          slot = 0;
        } else {
          const int64_t i = (int64_t)__umul64hi(b.x0, (uint64_t)n_set);
          slot = i < keep ? pos_list[n_pos - keep + i] : p.first_fresh + (i - keep);
        }
      }
      const int64_t r = phys_row(slot, p.head, p.cap);
      len = length[r];
      out_idx[j] = (int32_t)slot;
      out_adv[j] = advantage[r];
      out_len[j] = (int32_t)len;
      out_age[j] = p.cur_version - version[r];
    }
    int64_t total;
    if (p.layout == RB_LAYOUT_PACKED) {
      const int64_t ex = block_exclusive_scan<kDrawThreads>(len, &total, lds);
      if (j < p.n_draw) cu_seqlens[j + 1] = (int32_t)(carry + ex + len);
      carry += total;
    } else {
      const int64_t v = len < p.l_max ? len : p.l_max;
      block_exclusive_scan<kDrawThreads>(v, &total, lds);
      if (j < p.n_draw) cu_seqlens[j + 1] = (int32_t)((j + 1) * p.l_max);
      valid += total;
    }
  }
  if (threadIdx.x == 0) {
    if (p.layout == RB_LAYOUT_PACKED) {
      int64_t v = carry - p.token_begin;
      v = v < 0 ? 0 : (v > p.max_tokens ? p.max_tokens : v);
      *n_tokens = v;
      *stream_total = carry;
    } else {
      *n_tokens = valid;
      *stream_total = valid;
    }
  }
}

__global__ void __launch_bounds__(256) gather_packed_kernel(
    int64_t n_draw, int64_t head, int64_t cap, int64_t token_begin, int64_t max_tokens,
    const int64_t* __restrict__ stream_total, const int32_t* __restrict__ cu_seqlens,
    const int32_t* __restrict__ idx, const int64_t* __restrict__ arena_off,
    const int32_t* __restrict__ arena_tokens, const float* __restrict__ arena_old,
    int32_t* __restrict__ tokens, float* __restrict__ old_logp, int32_t* __restrict__ seq) {
  const int64_t total = *stream_total;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < max_tokens;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int64_t pos = token_begin + t;
    if (pos < total) {
      // largest j with cu_seqlens[j] <= pos (lengths are >= 1)
      int64_t lo = 0, hi = n_draw;  // invariant: cu[lo] <= pos < cu[hi]
      while (hi - lo > 1) {
        const int64_t mid = (lo + hi) >> 1;
        if (cu_seqlens[mid] <= pos) lo = mid; else hi = mid;
      }
      const int64_t src = arena_off[phys_row(idx[lo], head, cap)] + (pos - cu_seqlens[lo]);
      tokens[t] = arena_tokens[src];
      old_logp[t] = arena_old[src];
      seq[t] = (int32_t)lo;
    } else {
      tokens[t] = 0;
      old_logp[t] = 0.0f;
      seq[t] = -1;
    }
  }
}

// Padded rows: draw j fills row j of [n_draw, l_max] (positions past the
// record's length: token 0, log-prob 0, seq -1).  kVec: four positions per
// thread with 16-byte stores (l_max % 4 == 0, rows 16-byte aligned); the
// arena is read with 4-byte loads, its rows start anywhere.
template <bool kVec>
__global__ void __launch_bounds__(256) gather_padded_kernel(
    int64_t l_max, int64_t head, int64_t cap, const int32_t* __restrict__ idx,
    const int32_t* __restrict__ len, const int64_t* __restrict__ arena_off,
    const int32_t* __restrict__ arena_tokens, const float* __restrict__ arena_old,
    int32_t* __restrict__ tokens, float* __restrict__ old_logp, int32_t* __restrict__ seq) {
  const int64_t j = blockIdx.x;
  const int64_t n = len[j] < l_max ? len[j] : l_max;
  const int64_t off = arena_off[phys_row(idx[j], head, cap)];
  int32_t* tok_row = tokens + j * l_max;
  float* old_row = old_logp + j * l_max;
  int32_t* seq_row = seq + j * l_max;
  if constexpr (kVec) {
    for (int64_t p = ((int64_t)blockIdx.y * blockDim.x + threadIdx.x) * 4; p < l_max;
         p += (int64_t)gridDim.y * blockDim.x * 4) {
      int4 tk;
      float4 ol;
      int4 sq;
      int32_t* tkp = &tk.x;
      float* olp = &ol.x;
      int32_t* sqp = &sq.x;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool in = p + i < n;
        tkp[i] = in ? arena_tokens[off + p + i] : 0;
        olp[i] = in ? arena_old[off + p + i] : 0.0f;
        sqp[i] = in ? (int32_t)j : -1;
      }
      *reinterpret_cast<int4*>(tok_row + p) = tk;
      *reinterpret_cast<float4*>(old_row + p) = ol;
      *reinterpret_cast<int4*>(seq_row + p) = sq;
    }
  } else {
    for (int64_t p = (int64_t)blockIdx.y * blockDim.x + threadIdx.x; p < l_max;
         p += (int64_t)gridDim.y * blockDim.x) {
      if (p < n) {
        tok_row[p] = arena_tokens[off + p];
        old_row[p] = arena_old[off + p];
        seq_row[p] = (int32_t)j;
      } else {
        tok_row[p] = 0;
        old_row[p] = 0.0f;
        seq_row[p] = -1;
      }
    }
  }
}

}  // namespace

size_t rbp::sample_gather_ws(int64_t capacity) {
  const int64_t nb = ceil_div(capacity < 1 ? 1 : capacity, kSlotsPerBlock);
  WsCarver c(nullptr);
  c.take<int32_t>(nb);
  c.take<int32_t>(nb);
  c.take<int32_t>(capacity < 1 ? 1 : capacity);
  c.take<int64_t>(4);
  c.take<uint64_t>(capacity < 1 ? 1 : capacity);
  c.take<int64_t>(nb);
  c.take<int64_t>(nb);
  c.take<SelState>(1);
  return align_up(c.used, 256);
}

extern "C" int rb_sample_gather(const rb_records* rec, const rb_sample_cfg* cfg,
                                const rb_batch* out, void* ws, size_t ws_bytes,
                                void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(rec && cfg && out, RBP_EINVAL, "rb_sample_gather: null struct pointer");
  RBP_REQUIRE(rec->capacity >= 1 && rec->n_live >= 1 && rec->n_live <= rec->capacity,
              RBP_EINVAL, "rb_sample_gather: need 1 <= n_live <= capacity (got %lld, %lld)",
              (long long)rec->n_live, (long long)rec->capacity);
  RBP_REQUIRE(rec->capacity <= INT32_MAX, RBP_EINVAL,
              "rb_sample_gather: capacity above 2^31-1");
  RBP_REQUIRE(rec->head >= 0 && rec->head < rec->capacity, RBP_EINVAL,
              "rb_sample_gather: head outside [0, capacity)");
  RBP_REQUIRE(rec->arena_off && rec->length && rec->reward && rec->advantage &&
                  rec->version && rec->arena_tokens && rec->arena_old_logp,
              RBP_EINVAL, "rb_sample_gather: null record array");
  RBP_REQUIRE(cfg->mode >= RB_UNIFORM && cfg->mode <= RB_UNUSED_FIRST, RBP_EINVAL,
              "rb_sample_gather: unknown mode %d", cfg->mode);
  const bool no_replace = cfg->mode == RB_NO_REPLACE || cfg->mode == RB_UNUSED_FIRST;
  RBP_REQUIRE(!no_replace || cfg->n_draw <= rec->n_live, RBP_EINVAL,
              "rb_sample_gather: %lld draws without replacement from %lld records",
              (long long)cfg->n_draw, (long long)rec->n_live);
  RBP_REQUIRE(cfg->mode != RB_UNUSED_FIRST || rec->use_count != nullptr, RBP_EINVAL,
              "rb_sample_gather: RB_UNUSED_FIRST needs use_count");
  RBP_REQUIRE(cfg->layout == RB_LAYOUT_PACKED || cfg->layout == RB_LAYOUT_PADDED, RBP_EINVAL,
              "rb_sample_gather: unknown layout %d", cfg->layout);
  RBP_REQUIRE(cfg->n_draw >= 1 && cfg->n_draw <= (1 << 20), RBP_EINVAL,
              "rb_sample_gather: n_draw %lld outside [1, 2^20]", (long long)cfg->n_draw);
  RBP_REQUIRE(cfg->p_pos_q32 <= (1ull << 32), RBP_EINVAL,
              "rb_sample_gather: p_pos_q32 above 2^32");
  RBP_REQUIRE(cfg->n_fresh >= 0 && cfg->n_pos_keep >= 0, RBP_EINVAL,
              "rb_sample_gather: negative n_fresh / n_pos_keep");
  if (cfg->layout == RB_LAYOUT_PACKED) {
    RBP_REQUIRE(cfg->max_tokens >= 1 && cfg->token_begin >= 0, RBP_EINVAL,
                "rb_sample_gather: packed layout needs max_tokens >= 1, token_begin >= 0");
  } else {
    RBP_REQUIRE(cfg->l_max >= 1 && cfg->n_draw * cfg->l_max <= INT32_MAX, RBP_EINVAL,
                "rb_sample_gather: padded layout needs l_max >= 1 and n_draw * l_max < 2^31");
  }
  RBP_REQUIRE(out->idx && out->adv && out->len && out->age && out->cu_seqlens && out->tokens &&
                  out->old_logp && out->seq_of_token && out->n_tokens,
              RBP_EINVAL, "rb_sample_gather: null output array");
  const size_t need = rbp::sample_gather_ws(rec->capacity);
  RBP_REQUIRE(ws && ws_bytes >= need, RBP_EWORKSPACE,
              "rb_sample_gather: workspace needs %zu bytes, got %zu", need, ws_bytes);

  hipStream_t s = rbp::as_stream(stream);
  const int64_t nb_cap = rbp::ceil_div(rec->capacity, kSlotsPerBlock);
  rbp::WsCarver c(ws);
  int32_t* counts = c.take<int32_t>(nb_cap);
  int32_t* offsets = c.take<int32_t>(nb_cap);
  int32_t* pos_list = c.take<int32_t>(rec->capacity);
  int64_t* meta = c.take<int64_t>(4);
  uint64_t* keys = c.take<uint64_t>(rec->capacity);
  int64_t* sel_counts = c.take<int64_t>(nb_cap);
  int64_t* sel_offsets = c.take<int64_t>(nb_cap);
  SelState* sel_state = c.take<SelState>(1);

  DrawParams p{};
  p.mode = cfg->mode;
  p.layout = cfg->layout;
  p.seed = cfg->seed;
  p.step = cfg->step;
  p.p_q32 = cfg->p_pos_q32;
  p.n_draw = cfg->n_draw;
  p.n_live = rec->n_live;
  p.head = rec->head;
  p.cap = rec->capacity;
  p.first_fresh = rec->n_live - cfg->n_fresh;
  if (p.first_fresh < 0) p.first_fresh = 0;
  p.n_pos_keep = cfg->n_pos_keep;
  p.cur_version = cfg->cur_version;
  p.max_tokens = cfg->max_tokens;
  p.token_begin = cfg->token_begin;
  p.l_max = cfg->l_max;

  if (no_replace) {
    const int64_t n = rec->n_live;
    int64_t kb = rbp::ceil_div(n, 256);
    if (kb > 4096) kb = 4096;
    hipLaunchKernelGGL(slot_key_kernel, dim3(kb), dim3(256), 0, s, cfg->seed, cfg->step, n,
                       rec->head, rec->capacity,
                       cfg->mode == RB_UNUSED_FIRST ? rec->use_count : nullptr, keys);
    hipLaunchKernelGGL(select_init_kernel, dim3(1), dim3(256), 0, s, sel_state, cfg->n_draw);
    for (int pass = 0; pass < 8; ++pass) {
      hipLaunchKernelGGL(select_hist_kernel, dim3(kb), dim3(256), 0, s, keys, n, pass,
                         sel_state);
      hipLaunchKernelGGL(select_digit_kernel, dim3(1), dim3(256), 0, s, pass, sel_state);
    }
    const int64_t nb = rbp::ceil_div(n, kSlotsPerBlock);
    hipLaunchKernelGGL(sel_count_kernel, dim3(nb), dim3(kCountThreads), 0, s, keys, n, sel_state,
                       sel_counts);
    hipLaunchKernelGGL(sel_scan_kernel, dim3(1), dim3(1024), 0, s, sel_counts, sel_offsets, nb);
    hipLaunchKernelGGL(sel_compact_kernel, dim3(nb), dim3(kCountThreads), 0, s, keys, n,
                       sel_state, sel_offsets, pos_list);
  } else if (cfg->mode != RB_UNIFORM) {
    // positives over all live slots (mixture) or over the non-fresh ones (retention)
    const int64_t n_range = cfg->mode == RB_POS_MIX ? rec->n_live : p.first_fresh;
    const int64_t nb = rbp::ceil_div(n_range > 0 ? n_range : 1, kSlotsPerBlock);
    hipLaunchKernelGGL(pos_count_kernel, dim3(nb), dim3(kCountThreads), 0, s, rec->reward,
                       rec->head, rec->capacity, n_range, counts);
    hipLaunchKernelGGL(pos_scan_kernel, dim3(1), dim3(1024), 0, s, counts, offsets, nb, meta);
    hipLaunchKernelGGL(pos_compact_kernel, dim3(nb), dim3(kCountThreads), 0, s, rec->reward,
                       rec->head, rec->capacity, n_range, offsets, pos_list);
  }
  hipLaunchKernelGGL(draw_kernel, dim3(1), dim3(kDrawThreads), 0, s, p, meta, pos_list,
                     rec->length, rec->advantage, rec->version, out->idx, out->adv, out->len,
                     out->age, out->cu_seqlens, out->n_tokens, meta + 1);
  if (cfg->layout == RB_LAYOUT_PACKED) {
    int64_t blocks = rbp::ceil_div(cfg->max_tokens, 256);
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(gather_packed_kernel, dim3(blocks), dim3(256), 0, s, cfg->n_draw,
                       rec->head, rec->capacity, cfg->token_begin, cfg->max_tokens, meta + 1,
                       out->cu_seqlens, out->idx, rec->arena_off, rec->arena_tokens,
                       rec->arena_old_logp, out->tokens, out->old_logp, out->seq_of_token);
  } else {
    const bool vec = cfg->l_max % 4 == 0 &&
                     ((reinterpret_cast<uintptr_t>(out->tokens) |
                       reinterpret_cast<uintptr_t>(out->old_logp) |
                       reinterpret_cast<uintptr_t>(out->seq_of_token)) & 15) == 0;
    int64_t by = rbp::ceil_div(cfg->l_max, vec ? 1024 : 256);
    if (by > 64) by = 64;
    hipLaunchKernelGGL(vec ? gather_padded_kernel<true> : gather_padded_kernel<false>,
                       dim3(cfg->n_draw, by), dim3(256), 0, s, cfg->l_max, rec->head,
                       rec->capacity, out->idx, out->len, rec->arena_off, rec->arena_tokens,
                       rec->arena_old_logp, out->tokens, out->old_logp,
                       out->seq_of_token);
  }
  RBP_CHECK_LAUNCH("rb_sample_gather");
  return RBP_OK;
}
