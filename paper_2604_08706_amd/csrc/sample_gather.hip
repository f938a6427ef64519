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
//   [without replacement] slot_key -> select_top -> select_cand ->
//       select_rest -> sel_count -> sel_scan -> sel_compact : an MSD radix
//       select (8-bit digits) finds the n_draw-th smallest 64-bit slot key K
//       exactly -- the top digit from per-block histograms of every key, the
//       seven lower ones by one block over the keys that share the top digit
//       -- then the slots with a key below K (and the first ties in slot
//       order) are listed ascending;
//   draw     : one thread per draw; Philox4x64-10 block -> slot; per-draw
//              outputs; scan of lengths -> cu_seqlens, n_tokens (one block
//              up to 1024 draws, else draw_rows -> draw_scan -> draw_cu);
//   gather   : one block column per draw (packed: the part of its sequence
//              inside the window; padded: its l_max row); coalesced copies
//              from the token arena.
// Everything is integer work or a bit-exact copy of stored floats.

#include <atomic>
#include <mutex>

#include "rbp_internal.h"

namespace {

constexpr int kSlotsPerBlock = 1024;  // compaction granule
constexpr int kCountThreads = 256;    // 4 slots per thread
constexpr int kDrawThreads = 1024;  // single-block draw pass, up to this many draws
constexpr int kRowThreads = 256;    // draws per block beyond that
constexpr int kMaxRowBlocks = (1 << 20) / kRowThreads;

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

constexpr int kKeyBlocks = 256;   // key kernel blocks (at most): key segments; a power of 2
constexpr int kKeyThreads = 1024;
constexpr int kTopThreads = 1024;
constexpr int kRestThreads = 1024;
constexpr int kRestRegKeys = 16;  // candidates per thread held in registers

// Radix-select state: the key digits fixed so far and how many keys still to
// be taken among those sharing them.
struct SelState {
  uint64_t prefix;
  int64_t need;
};

// Key segment b of n keys split over n_seg blocks: [b * per, min(n, (b+1) * per)).
__device__ __forceinline__ int64_t seg_len(int64_t n, int64_t n_seg) {
  return (n + n_seg - 1) / n_seg;
}

// Key of slot s: the top 63 bits of word 0 of the Philox block with counter
// (s, step, 1, 0); for never-used-first, bit 63 set when the slot was used.
// Block b keys segment b and writes the histogram of the top digit (bits
// 56..63) of its keys to row b of `top_hist`: no global atomics, so the 256
// bins are not contended by every block.
__global__ void __launch_bounds__(kKeyThreads) slot_key_kernel(
    uint64_t seed, uint64_t step, int64_t n_live, int64_t head, int64_t cap,
    const int32_t* __restrict__ use_count, uint64_t* __restrict__ keys,
    uint32_t* __restrict__ top_hist) {
  __shared__ uint32_t h[256];
  if (threadIdx.x < 256) h[threadIdx.x] = 0u;
  __syncthreads();
  const int64_t per = seg_len(n_live, gridDim.x);
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < n_live ? lo + per : n_live;
  for (int64_t s = lo + threadIdx.x; s < hi; s += kKeyThreads) {
    uint64_t k = philox4x64_10((uint64_t)s, step, 1, 0, seed, 0).x0 >> 1;
    if (use_count != nullptr && use_count[phys_row(s, head, cap)] > 0) k |= 1ull << 63;
    keys[s] = k;
    atomicAdd(&h[k >> 56], 1u);
  }
  __syncthreads();
  if (threadIdx.x < 256) top_hist[blockIdx.x * 256 + threadIdx.x] = h[threadIdx.x];
}

// Bin t of the block holding the need-th smallest remaining key: the one
// thread whose exclusive prefix is below `need` and inclusive prefix reaches
// it (empty bins never qualify).
__device__ __forceinline__ bool holds_need(int64_t excl, int64_t count, int64_t need) {
  return excl < need && need <= excl + count;
}

// One block: sums the per-segment top-digit histograms (four threads per
// bin) and picks the top digit.
__global__ void __launch_bounds__(kTopThreads) select_top_kernel(
    const uint32_t* __restrict__ top_hist, int32_t n_seg, int64_t n_draw,
    SelState* __restrict__ st) {
  __shared__ uint32_t part[kTopThreads / 256][256];
  __shared__ int64_t lds[kTopThreads / 64];
  const int bin = threadIdx.x & 255, q = threadIdx.x >> 8;
  uint32_t c = 0u;
#pragma unroll 8
  for (int32_t b = q; b < n_seg; b += kTopThreads / 256) c += top_hist[b * 256 + bin];
  part[q][bin] = c;
  __syncthreads();
  int64_t v = 0;
  if (threadIdx.x < 256)
    for (int i = 0; i < kTopThreads / 256; ++i) v += part[i][bin];
  int64_t total;
  const int64_t excl = block_exclusive_scan<kTopThreads>(v, &total, lds);
  if (threadIdx.x < 256 && holds_need(excl, v, n_draw)) {
    st->prefix = (uint64_t)bin << 56;
    st->need = n_draw - excl;
  }
}

// Block b lists the keys of segment b whose top digit is the selected one at
// the start of the segment's stretch of `cand` (order free: only their digit
// histograms are taken), and their number in cand_cnt[b].  One LDS atomic per
// wave, no global ones.
__global__ void __launch_bounds__(kKeyThreads) select_cand_kernel(
    const uint64_t* __restrict__ keys, int64_t n, const SelState* __restrict__ st,
    uint64_t* __restrict__ cand, uint32_t* __restrict__ cand_cnt) {
  __shared__ uint32_t cnt;
  if (threadIdx.x == 0) cnt = 0u;
  __syncthreads();
  const uint64_t top = st->prefix >> 56;
  const int lane = threadIdx.x & 63;
  const int64_t per = seg_len(n, gridDim.x);
  const int64_t lo = (int64_t)blockIdx.x * per;
  const int64_t hi = lo + per < n ? lo + per : n;
  for (int64_t base = lo; base < hi; base += kKeyThreads) {
    const int64_t s = base + threadIdx.x;
    const uint64_t k = s < hi ? keys[s] : 0ull;
    const bool take = s < hi && (k >> 56) == top;
    const uint64_t m = __ballot(take);
    if (m == 0ull) continue;
    uint32_t at = 0u;
    if (lane == 0) at = atomicAdd(&cnt, (uint32_t)__popcll(m));
    at = __shfl(at, 0, 64);
    if (take) cand[lo + at + __popcll(m & ((1ull << lane) - 1ull))] = k;
  }
  __syncthreads();
  if (threadIdx.x == 0) cand_cnt[blockIdx.x] = cnt;
}

// One block: the lower digits, most significant first, over the candidates
// only (the first kRestThreads * kRestRegKeys of them held in registers, any
// further ones re-read each pass), until at most kRestThreads keys share the
// prefix; those are then ranked directly, each thread counting the survivors
// below and up to its own.  Integer counts only: the result does not depend
// on the order of any addition.  Leaves the exact need-th smallest key in
// `prefix` and the number of its ties still to be taken in `need`.
__global__ void __launch_bounds__(kRestThreads) select_rest_kernel(
    const uint64_t* __restrict__ cand, const uint32_t* __restrict__ cand_cnt, int32_t n_seg,
    int64_t n, SelState* __restrict__ st) {
  __shared__ uint32_t h[256];
  __shared__ int64_t lds[kRestThreads / 64];
  __shared__ int64_t seg_start[kKeyBlocks + 1];
  __shared__ uint64_t surv[kRestThreads];
  __shared__ uint64_t s_prefix;
  __shared__ int64_t s_need, s_match;
  __shared__ uint32_t s_surv;
  const int64_t c = threadIdx.x < n_seg ? (int64_t)cand_cnt[threadIdx.x] : 0;
  int64_t nc;
  const int64_t excl = block_exclusive_scan<kRestThreads>(c, &nc, lds);
  if (threadIdx.x < n_seg) seg_start[threadIdx.x] = excl;
  if (threadIdx.x == 0) {
    seg_start[n_seg] = nc;
    s_surv = 0u;
  }
  __syncthreads();
  const int64_t per = seg_len(n, n_seg);
  // candidate i (< nc) sits at entry i - seg_start[b] of segment b, the last
  // segment starting at or before i
  // (a fixed eight halvings over n_seg <= kKeyBlocks = 256 starts, so the
  // searches of a thread's candidates interleave)
  auto cand_pos = [&](int64_t i) {
    int lo = 0;
#pragma unroll
    for (int step = kKeyBlocks / 2; step > 0; step >>= 1) {
      const int m = lo + step;
      if (m < n_seg && seg_start[m] <= i) lo = m;
    }
    return lo * per + (i - seg_start[lo]);
  };
  // positions first, then all the loads together (nc >= 1: the selected
  // bucket holds the need-th key; indices past it re-read the last one)
  int64_t at[kRestRegKeys];
#pragma unroll
  for (int u = 0; u < kRestRegKeys; ++u) {
    const int64_t i = threadIdx.x + (int64_t)u * kRestThreads;
    at[u] = cand_pos(i < nc ? i : nc - 1);
  }
  uint64_t reg[kRestRegKeys];
#pragma unroll
  for (int u = 0; u < kRestRegKeys; ++u) reg[u] = cand[at[u]];
  // calls f(k) for every candidate k
  auto each_cand = [&](auto&& f) {
#pragma unroll
    for (int u = 0; u < kRestRegKeys; ++u)
      if (threadIdx.x + (int64_t)u * kRestThreads < nc) f(reg[u]);
    for (int64_t i = threadIdx.x + (int64_t)kRestRegKeys * kRestThreads; i < nc;
         i += kRestThreads)
      f(cand[cand_pos(i)]);
  };
  uint64_t prefix = st->prefix;
  int64_t need = st->need;
  int64_t n_match = nc;  // keys sharing the digits fixed so far
  int shift = 56;        // the prefix fixes the bits from `shift` up
  while (shift > 0 && n_match > kRestThreads) {
    shift -= 8;
    if (threadIdx.x < 256) h[threadIdx.x] = 0u;
    __syncthreads();
    const uint64_t hi = prefix >> (shift + 8);
    each_cand([&](uint64_t k) {
      if ((k >> (shift + 8)) == hi) atomicAdd(&h[(k >> shift) & 255u], 1u);
    });
    __syncthreads();
    const int64_t v = threadIdx.x < 256 ? (int64_t)h[threadIdx.x] : 0;
    int64_t total;
    const int64_t ex = block_exclusive_scan<kRestThreads>(v, &total, lds);
    if (threadIdx.x < 256 && holds_need(ex, v, need)) {
      s_prefix = prefix | ((uint64_t)threadIdx.x << shift);
      s_need = need - ex;
      s_match = v;
    }
    __syncthreads();
    prefix = s_prefix;
    need = s_need;
    n_match = s_match;
  }
  if (shift > 0) {
    // at most kRestThreads survivors: list them (order free), then the one
    // with `need - 1` survivors strictly below it and at least `need` up to
    // it is the key; equal keys all write the same values
    const uint64_t hi = prefix >> shift;
    each_cand([&](uint64_t k) {
      if ((k >> shift) == hi) {
        const uint32_t i = atomicAdd(&s_surv, 1u);  // < n_match <= kRestThreads
        if (i < kRestThreads) surv[i] = k;
      }
    });
    __syncthreads();
    if (threadIdx.x < n_match) {
      const uint64_t mine = surv[threadIdx.x];
      int64_t less = 0, leq = 0;
      for (int64_t i = 0; i < n_match; ++i) {
        const uint64_t o = surv[i];
        less += o < mine;
        leq += o <= mine;
      }
      if (less < need && need <= leq) {
        s_prefix = mine;
        s_need = need - less;
      }
    }
    __syncthreads();
    prefix = s_prefix;
    need = s_need;
  }
  if (threadIdx.x == 0) {
    st->prefix = prefix;
    st->need = need;
  }
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

// Per-call constants of the draws: the positives listed by the count/scan
// pass, the retained positives and the size of the retained set.
struct DrawSet {
  int64_t n_pos, keep, n_set;
};

__device__ __forceinline__ DrawSet draw_set(const DrawParams& p,
                                            const int64_t* __restrict__ meta) {
  DrawSet d;
  d.n_pos = (p.mode == RB_POS_MIX || p.mode == RB_POS_RETAIN) ? meta[0] : 0;
  // retained set: the newest `keep` positives older than the fresh part, then
  // the fresh part [first_fresh, n_live)
  d.keep = d.n_pos < p.n_pos_keep ? d.n_pos : p.n_pos_keep;
  d.n_set = d.keep + (p.n_live - p.first_fresh);
  return d;
}

// Slot of draw j: the Philox4x64-10 block with counter (j, step, 0, 0) picks
// it (or the j-th selected slot without replacement).
__device__ __forceinline__ int64_t draw_slot(const DrawParams& p, const DrawSet& d,
                                             const int32_t* __restrict__ pos_list, int64_t j) {
  if (p.mode == RB_NO_REPLACE || p.mode == RB_UNUSED_FIRST) return pos_list[j];
  const Block4 b = philox4x64_10((uint64_t)j, p.step, 0, 0, p.seed, 0);
  if (p.mode == RB_UNIFORM) return (int64_t)__umul64hi(b.x0, (uint64_t)p.n_live);
  if (p.mode == RB_POS_MIX) {
    if (d.n_pos > 0 && (b.x1 >> 32) < p.p_q32) return pos_list[__umul64hi(b.x0, (uint64_t)d.n_pos)];
    return (int64_t)__umul64hi(b.x0, (uint64_t)p.n_live);
  }
  if (d.n_set <= 0) return 0;
  const int64_t i = (int64_t)__umul64hi(b.x0, (uint64_t)d.n_set);
  return i < d.keep ? pos_list[d.n_pos - d.keep + i] : p.first_fresh + (i - d.keep);
}

// Per-draw outputs of draw j; returns its contribution to the stream (full
// length packed, min(length, l_max) padded).
__device__ __forceinline__ int64_t draw_one(const DrawParams& p, const DrawSet& d,
                                            const int32_t* __restrict__ pos_list,
                                            const int32_t* __restrict__ length,
                                            const float* __restrict__ advantage,
                                            const int32_t* __restrict__ version, int64_t j,
                                            int32_t* __restrict__ out_idx,
                                            float* __restrict__ out_adv,
                                            int32_t* __restrict__ out_len,
                                            int32_t* __restrict__ out_age) {
  const int64_t slot = draw_slot(p, d, pos_list, j);
  const int64_t r = phys_row(slot, p.head, p.cap);
  const int64_t len = length[r];
  out_idx[j] = (int32_t)slot;
  out_adv[j] = advantage[r];
  out_len[j] = (int32_t)len;
  out_age[j] = p.cur_version - version[r];
  return p.layout == RB_LAYOUT_PACKED ? len : (len < p.l_max ? len : p.l_max);
}

__device__ __forceinline__ void write_totals(const DrawParams& p, int64_t sum,
                                             int64_t* __restrict__ n_tokens,
                                             int64_t* __restrict__ stream_total) {
  if (p.layout == RB_LAYOUT_PACKED) {
    int64_t v = sum - p.token_begin;
    v = v < 0 ? 0 : (v > p.max_tokens ? p.max_tokens : v);
    *n_tokens = v;
  } else {
    *n_tokens = sum;
  }
  *stream_total = sum;
}

// Up to kDrawThreads draws: one block, one draw per thread, block scan of the
// lengths -> cu_seqlens, n_tokens.
__global__ void __launch_bounds__(kDrawThreads) draw_kernel(
    DrawParams p, const int64_t* __restrict__ meta, const int32_t* __restrict__ pos_list,
    const int32_t* __restrict__ length, const float* __restrict__ advantage,
    const int32_t* __restrict__ version, int32_t* __restrict__ out_idx,
    float* __restrict__ out_adv, int32_t* __restrict__ out_len, int32_t* __restrict__ out_age,
    int32_t* __restrict__ cu_seqlens, int64_t* __restrict__ n_tokens,
    int64_t* __restrict__ stream_total) {
  __shared__ int64_t lds[kDrawThreads / 64];
  const DrawSet d = draw_set(p, meta);
  const int64_t j = threadIdx.x;
  const int64_t v = j < p.n_draw ? draw_one(p, d, pos_list, length, advantage, version, j,
                                            out_idx, out_adv, out_len, out_age)
                                 : 0;
  int64_t total;
  const int64_t ex = block_exclusive_scan<kDrawThreads>(v, &total, lds);
  if (j == 0) cu_seqlens[0] = 0;
  if (j < p.n_draw)
    cu_seqlens[j + 1] = (int32_t)(p.layout == RB_LAYOUT_PACKED ? ex + v : (j + 1) * p.l_max);
  if (j == 0) write_totals(p, total, n_tokens, stream_total);
}

// More draws: blocks of kRowThreads draws write the per-draw outputs and
// their block sums; one block scans the sums; then each block writes its
// cu_seqlens.  Many blocks keep the scattered record reads spread over the
// chip.
__global__ void __launch_bounds__(kRowThreads) draw_rows_kernel(
    DrawParams p, const int64_t* __restrict__ meta, const int32_t* __restrict__ pos_list,
    const int32_t* __restrict__ length, const float* __restrict__ advantage,
    const int32_t* __restrict__ version, int32_t* __restrict__ out_idx,
    float* __restrict__ out_adv, int32_t* __restrict__ out_len, int32_t* __restrict__ out_age,
    int64_t* __restrict__ blk_sum) {
  __shared__ int64_t lds[kRowThreads / 64];
  const DrawSet d = draw_set(p, meta);
  const int64_t j = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  const int64_t v = j < p.n_draw ? draw_one(p, d, pos_list, length, advantage, version, j,
                                            out_idx, out_adv, out_len, out_age)
                                 : 0;
  int64_t total;
  block_exclusive_scan<kRowThreads>(v, &total, lds);
  if (threadIdx.x == 0) blk_sum[blockIdx.x] = total;
}

__global__ void __launch_bounds__(1024) draw_scan_kernel(DrawParams p,
                                                         const int64_t* __restrict__ blk_sum,
                                                         int64_t* __restrict__ blk_off, int64_t nb,
                                                         int64_t* __restrict__ n_tokens,
                                                         int64_t* __restrict__ stream_total) {
  __shared__ int64_t lds[1024 / 64];
  int64_t carry = 0;
  for (int64_t base = 0; base < nb; base += 1024) {
    const int64_t i = base + threadIdx.x;
    const int64_t v = i < nb ? blk_sum[i] : 0;
    int64_t total;
    const int64_t ex = block_exclusive_scan<1024>(v, &total, lds);
    if (i < nb) blk_off[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) write_totals(p, carry, n_tokens, stream_total);
}

__global__ void __launch_bounds__(kRowThreads) draw_cu_kernel(
    DrawParams p, const int32_t* __restrict__ out_len, const int64_t* __restrict__ blk_off,
    int32_t* __restrict__ cu_seqlens) {
  __shared__ int64_t lds[kRowThreads / 64];
  const int64_t j = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  const int64_t v = j < p.n_draw ? (int64_t)out_len[j] : 0;
  int64_t total;
  const int64_t ex = block_exclusive_scan<kRowThreads>(v, &total, lds);
  if (j == 0) cu_seqlens[0] = 0;
  if (j < p.n_draw)
    cu_seqlens[j + 1] = (int32_t)(p.layout == RB_LAYOUT_PACKED ? blk_off[blockIdx.x] + ex + v
                                                               : (j + 1) * p.l_max);
}

// Block (j, y) copies the tokens of draw j that fall in the window
// [token_begin, token_begin + max_tokens) of the packed stream, rows y
// splitting long sequences; every block also takes its share of the window
// positions past the end of the stream, which are padded.
__global__ void __launch_bounds__(256) gather_packed_kernel(
    int64_t head, int64_t cap, int64_t token_begin, int64_t max_tokens,
    const int64_t* __restrict__ stream_total, const int32_t* __restrict__ cu_seqlens,
    const int32_t* __restrict__ idx, const int64_t* __restrict__ arena_off,
    const int32_t* __restrict__ arena_tokens, const float* __restrict__ arena_old,
    int32_t* __restrict__ tokens, float* __restrict__ old_logp, int32_t* __restrict__ seq) {
  const int64_t win_end = token_begin + max_tokens;
  const int64_t total = *stream_total;
  const int64_t n_blk = (int64_t)gridDim.x * gridDim.y;
  const int64_t blk = (int64_t)blockIdx.x * gridDim.y + blockIdx.y;
  for (int64_t pos = (total > token_begin ? total : token_begin) + blk * 256 + threadIdx.x;
       pos < win_end; pos += n_blk * 256) {
    const int64_t t = pos - token_begin;
    tokens[t] = 0;
    old_logp[t] = 0.0f;
    seq[t] = -1;
  }
  const int64_t j = blockIdx.x;
  const int64_t c0 = cu_seqlens[j], c1 = cu_seqlens[j + 1];
  const int64_t lo = c0 > token_begin ? c0 : token_begin;
  const int64_t hi = c1 < win_end ? c1 : win_end;
  if (lo >= hi) return;
  const int64_t src = arena_off[phys_row(idx[j], head, cap)] - c0;  // + stream position
  for (int64_t pos = lo + (int64_t)blockIdx.y * 256 + threadIdx.x; pos < hi;
       pos += (int64_t)gridDim.y * 256) {
    const int64_t t = pos - token_begin;
    tokens[t] = arena_tokens[src + pos];
    old_logp[t] = arena_old[src + pos];
    seq[t] = (int32_t)j;
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
  c.take<uint32_t>(kKeyBlocks * 256);
  c.take<uint32_t>(kKeyBlocks);
  c.take<uint64_t>(capacity < 1 ? 1 : capacity);
  c.take<int64_t>(kMaxRowBlocks);
  c.take<int64_t>(kMaxRowBlocks);
  return align_up(c.used, 256);
}

namespace {

// Everything rb_sample_gather does after clearing the error text: argument
// checks, then the device pipeline with `ws` as its workspace.
int sample_gather(const rb_records* rec, const rb_sample_cfg* cfg, const rb_batch* out, void* ws,
                  size_t ws_bytes, void* stream) {
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
  uint32_t* top_hist = c.take<uint32_t>(kKeyBlocks * 256);
  uint32_t* cand_cnt = c.take<uint32_t>(kKeyBlocks);
  uint64_t* cand = c.take<uint64_t>(rec->capacity);
  int64_t* blk_sum = c.take<int64_t>(kMaxRowBlocks);
  int64_t* blk_off = c.take<int64_t>(kMaxRowBlocks);

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
    int64_t kb = rbp::ceil_div(n, 2048);
    if (kb > kKeyBlocks) kb = kKeyBlocks;
    hipLaunchKernelGGL(slot_key_kernel, dim3(kb), dim3(kKeyThreads), 0, s, cfg->seed, cfg->step,
                       n, rec->head, rec->capacity,
                       cfg->mode == RB_UNUSED_FIRST ? rec->use_count : nullptr, keys, top_hist);
    hipLaunchKernelGGL(select_top_kernel, dim3(1), dim3(kTopThreads), 0, s, top_hist,
                       (int32_t)kb, cfg->n_draw, sel_state);
    hipLaunchKernelGGL(select_cand_kernel, dim3(kb), dim3(kKeyThreads), 0, s, keys, n,
                       sel_state, cand, cand_cnt);
    hipLaunchKernelGGL(select_rest_kernel, dim3(1), dim3(kRestThreads), 0, s, cand, cand_cnt,
                       (int32_t)kb, n, sel_state);
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
  if (cfg->n_draw <= kDrawThreads) {
    hipLaunchKernelGGL(draw_kernel, dim3(1), dim3(kDrawThreads), 0, s, p, meta, pos_list,
                       rec->length, rec->advantage, rec->version, out->idx, out->adv, out->len,
                       out->age, out->cu_seqlens, out->n_tokens, meta + 1);
  } else {
    const int64_t nb = rbp::ceil_div(cfg->n_draw, kRowThreads);
    hipLaunchKernelGGL(draw_rows_kernel, dim3(nb), dim3(kRowThreads), 0, s, p, meta, pos_list,
                       rec->length, rec->advantage, rec->version, out->idx, out->adv, out->len,
                       out->age, blk_sum);
    hipLaunchKernelGGL(draw_scan_kernel, dim3(1), dim3(1024), 0, s, p, blk_sum, blk_off, nb,
                       out->n_tokens, meta + 1);
    hipLaunchKernelGGL(draw_cu_kernel, dim3(nb), dim3(kRowThreads), 0, s, p, out->len, blk_off,
                       out->cu_seqlens);
  }
  if (cfg->layout == RB_LAYOUT_PACKED) {
    // about 256 window positions per block
    int64_t by = rbp::ceil_div(cfg->max_tokens, cfg->n_draw * 256);
    if (by > 64) by = 64;
    hipLaunchKernelGGL(gather_packed_kernel, dim3(cfg->n_draw, by), dim3(256), 0, s,
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

// Workspace of rb_sample_gather_noalloc: one array per device, held from
// module load until the process ends.  In host code `scratch` names a
// host-side stand-in; the device address comes from hipGetSymbolAddress.
constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];
std::mutex g_scratch_lock;

// The current device's address of `scratch`, resolved on the first call on
// that device (with the device current) and kept.
int scratch_addr(void** addr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  RBP_REQUIRE(e == hipSuccess, RBP_EHIP, "rb_sample_gather_noalloc: hipGetDevice: %s",
              hipGetErrorString(e));
  RBP_REQUIRE(dev >= 0 && dev < kMaxDevices, RBP_EUNSUPPORTED,
              "rb_sample_gather_noalloc: device %d beyond the %d the library tracks", dev,
              kMaxDevices);
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> g(g_scratch_lock);
    p = g_scratch_addr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      RBP_REQUIRE(e == hipSuccess && p != nullptr, RBP_EHIP,
                  "rb_sample_gather_noalloc: hipGetSymbolAddress(scratch) on device %d: %s",
                  dev, hipGetErrorString(e));
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *addr = p;
  return RBP_OK;
}

}  // namespace

extern "C" int rb_sample_gather(const rb_records* rec, const rb_sample_cfg* cfg,
                                const rb_batch* out, void* ws, size_t ws_bytes,
                                void* stream) {
  rbp::clear_error();
  return sample_gather(rec, cfg, out, ws, ws_bytes, stream);
}

extern "C" int rb_sample_gather_noalloc(const rb_records* rec, const rb_sample_cfg* cfg,
                                        const rb_batch* out, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(rec, RBP_EINVAL, "rb_sample_gather_noalloc: null record table");
  RBP_REQUIRE(rec->capacity >= 1 && rec->capacity <= INT32_MAX, RBP_EINVAL,
              "rb_sample_gather_noalloc: capacity %lld outside [1, 2^31-1]",
              (long long)rec->capacity);
  const size_t need = rbp::sample_gather_ws(rec->capacity);
  RBP_REQUIRE(need <= kScratchBytes, RBP_EWORKSPACE,
              "rb_sample_gather_noalloc: a record table of capacity %lld needs %zu bytes of "
              "workspace, more than the %zu-byte static scratch (use rb_sample_gather with a "
              "caller workspace)",
              (long long)rec->capacity, need, kScratchBytes);
  void* ws = nullptr;
  const int st = scratch_addr(&ws);
  if (st != RBP_OK) return st;
  return sample_gather(rec, cfg, out, ws, kScratchBytes, stream);
}
