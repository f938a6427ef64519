// Buffer maintenance: FIFO insertion of generated groups (rb_push),
// per-record usage bookkeeping (rb_note_use) and the histograms of the buffer
// statistics (rb_hist_accumulate).
//
// Paper: the buffer holds the N most recent rollouts; a push into a full
// buffer evicts the oldest one and sampling never removes (App. B
// "BufferStructure"); advantages are computed once, when a group is generated
// (App. D.2).  Steps-since-last-use (App. D.3, "Metrics"): a rollout's first
// sample is "new", a later one gets the gradient steps since its previous
// sample, 0 for repeats inside one batch.  Sec. 3.2 reports the distributions
// of off-policiness (a sample's age), replay ratio (uses of a rollout over the
// run) and steps since last use.
//
// The record table is a ring: logical slot s is physical row (head + s) %
// capacity, and row r owns a fixed arena stretch of slot_tokens tokens, so an
// inserted record always overwrites the storage of the record it evicts.
// Everything here is integer work or a copy, except the advantage (fp32, the
// arithmetic of rb_group_advantage).

#include "group_advantage.h"
#include "rbp_internal.h"

namespace {

__device__ __forceinline__ int64_t ring_row(int64_t base, int64_t i, int64_t cap) {
  const int64_t r = base + i;
  return r >= cap ? r - cap : r;
}

// One thread per new group: advantages straight into the ring rows.
__global__ void __launch_bounds__(64) push_advantage_kernel(
    const float* __restrict__ reward, const int32_t* __restrict__ group_off, int32_t n_groups,
    int32_t ddof, float eps, int64_t base, int64_t cap, float* __restrict__ adv) {
  const int32_t g = blockIdx.x * 64 + threadIdx.x;
  if (g >= n_groups) return;
  rbp::group_advantage(reward, group_off[g], group_off[g + 1], ddof, eps,
                       [&](int32_t i, float a) { adv[ring_row(base, i, cap)] = a; });
}

// One thread per new record: the per-record fields of its row.
__global__ void __launch_bounds__(256) push_rows_kernel(
    int32_t n_new, int64_t base, int64_t cap, int64_t slot_tokens,
    const int32_t* __restrict__ length, const float* __restrict__ reward, int32_t version,
    int64_t* __restrict__ r_off, int32_t* __restrict__ r_len, float* __restrict__ r_reward,
    int32_t* __restrict__ r_version, int32_t* __restrict__ r_uses,
    int64_t* __restrict__ r_last) {
  const int32_t i = blockIdx.x * 256 + threadIdx.x;
  if (i >= n_new) return;
  const int64_t r = ring_row(base, i, cap);
  const int32_t len = length[i];
  r_off[r] = r * slot_tokens;
  r_len[r] = (int64_t)len < slot_tokens ? len : (int32_t)slot_tokens;
  r_reward[r] = reward[i];
  r_version[r] = version;
  if (r_uses != nullptr) r_uses[r] = 0;
  if (r_last != nullptr) r_last[r] = -1;
}

// Block row i copies record i's tokens and behaviour log-probs into its row's
// arena stretch (at most slot_tokens of them).
__global__ void __launch_bounds__(256) push_copy_kernel(
    int64_t base, int64_t cap, int64_t slot_tokens, const int32_t* __restrict__ length,
    const int64_t* __restrict__ src_off, const int32_t* __restrict__ tokens,
    const float* __restrict__ old_logp, int32_t* __restrict__ arena_tokens,
    float* __restrict__ arena_old) {
  const int32_t i = blockIdx.x;
  const int64_t r = ring_row(base, i, cap);
  int64_t n = length[i];
  if (n > slot_tokens) n = slot_tokens;
  const int64_t src = src_off[i], dst = r * slot_tokens;
  for (int64_t p = (int64_t)blockIdx.y * 256 + threadIdx.x; p < n;
       p += (int64_t)gridDim.y * 256) {
    arena_tokens[dst + p] = tokens[src + p];
    arena_old[dst + p] = old_logp[src + p];
  }
}

// Replay ratio of the records a push evicts (Sec. 3.2): new record i >= first
// overwrites a row that still holds a live record; its final use count goes
// to the histogram before push_rows_kernel resets it.
__global__ void __launch_bounds__(256) push_evict_kernel(int32_t n_new, int64_t first,
                                                         int64_t base, int64_t cap,
                                                         const int32_t* __restrict__ uses,
                                                         int32_t n_bins,
                                                         int64_t* __restrict__ hist) {
  const int64_t i = first + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n_new) return;
  int32_t u = uses[ring_row(base, i, cap)];
  u = u < 0 ? 0 : (u > n_bins - 1 ? n_bins - 1 : u);
  atomicAdd(reinterpret_cast<unsigned long long*>(hist + u), 1ull);
}

// ---- usage bookkeeping ------------------------------------------------------

__device__ __forceinline__ int64_t drawn_row(const int32_t* __restrict__ idx, int64_t j,
                                             int64_t head, int64_t cap) {
  return ring_row(head, idx[j], cap);
}

__global__ void __launch_bounds__(256) use_reset_kernel(const int32_t* __restrict__ idx,
                                                        int64_t n, int64_t head, int64_t cap,
                                                        int32_t* __restrict__ first) {
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256)
    first[drawn_row(idx, j, head, cap)] = INT32_MAX;
}

// first[row] = smallest draw index of the batch that took the row
__global__ void __launch_bounds__(256) use_first_kernel(const int32_t* __restrict__ idx,
                                                        int64_t n, int64_t head, int64_t cap,
                                                        int32_t* __restrict__ first) {
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256)
    atomicMin(&first[drawn_row(idx, j, head, cap)], (int32_t)j);
}

__global__ void __launch_bounds__(256) use_since_kernel(const int32_t* __restrict__ idx,
                                                        int64_t n, int64_t head, int64_t cap,
                                                        int64_t step,
                                                        const int32_t* __restrict__ first,
                                                        const int64_t* __restrict__ last,
                                                        int32_t* __restrict__ since) {
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n;
       j += (int64_t)gridDim.x * 256) {
    const int64_t r = drawn_row(idx, j, head, cap);
    const int64_t l = last[r];
    since[j] = first[r] < j ? 0 : (l < 0 ? -1 : (int32_t)(step - l));
  }
}

// use_count += draws of the row (integer atomics: the sum is order-free);
// the row's first draw stores the step.
__global__ void __launch_bounds__(256) use_update_kernel(const int32_t* __restrict__ idx,
                                                         int64_t n, int64_t head, int64_t cap,
                                                         int64_t step,
                                                         const int32_t* __restrict__ first,
                                                         int32_t* __restrict__ uses,
                                                         int64_t* __restrict__ last) {
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n;
       j += (int64_t)gridDim.x * 256) {
    const int64_t r = drawn_row(idx, j, head, cap);
    atomicAdd(&uses[r], 1);
    if (first[r] == j) last[r] = step;
  }
}

// ---- statistics ------------------------------------------------------------

constexpr int kHistMaxBins = 4096;

// Block histogram in LDS, then one integer atomic per non-empty bin.
__global__ void __launch_bounds__(256) hist_kernel(const int32_t* __restrict__ values, int64_t n,
                                                   int32_t lo, int32_t n_bins,
                                                   int64_t* __restrict__ hist) {
  __shared__ uint32_t h[kHistMaxBins];
  for (int b = threadIdx.x; b < n_bins; b += 256) h[b] = 0u;
  __syncthreads();
  for (int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (int64_t)gridDim.x * 256) {
    int64_t b = (int64_t)values[j] - lo;
    b = b < 0 ? 0 : (b > n_bins - 1 ? n_bins - 1 : b);
    atomicAdd(&h[b], 1u);
  }
  __syncthreads();
  for (int b = threadIdx.x; b < n_bins; b += 256)
    if (h[b] != 0u) atomicAdd(reinterpret_cast<unsigned long long*>(hist + b), (unsigned long long)h[b]);
}

}  // namespace

size_t rbp::note_use_ws(int64_t capacity) {
  return align_up(sizeof(int32_t) * (size_t)(capacity < 1 ? 1 : capacity), 256);
}

extern "C" int rb_push(rb_ring* ring, int32_t n_new, int32_t n_groups, const int32_t* group_off,
                       const int32_t* length, const int64_t* src_off, const float* reward,
                       int32_t version, const int32_t* tokens, const float* old_logp,
                       int32_t ddof, float eps, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(ring != nullptr, RBP_EINVAL, "rb_push: null ring");
  const int64_t cap = ring->capacity;
  RBP_REQUIRE(cap >= 1 && cap <= INT32_MAX, RBP_EINVAL, "rb_push: capacity outside [1, 2^31)");
  RBP_REQUIRE(ring->n_live >= 0 && ring->n_live <= cap, RBP_EINVAL,
              "rb_push: n_live outside [0, capacity]");
  RBP_REQUIRE(ring->head >= 0 && ring->head < cap, RBP_EINVAL, "rb_push: head outside [0, capacity)");
  RBP_REQUIRE(ring->slot_tokens >= 1, RBP_EINVAL, "rb_push: slot_tokens < 1");
  RBP_REQUIRE(n_new >= 1 && n_new <= cap, RBP_EINVAL, "rb_push: n_new %d outside [1, capacity]",
              n_new);
  RBP_REQUIRE(n_groups >= 1, RBP_EINVAL, "rb_push: n_groups < 1");
  RBP_REQUIRE(ddof == 0 || ddof == 1, RBP_EINVAL, "rb_push: ddof must be 0 or 1");
  RBP_REQUIRE(eps >= 0.0f, RBP_EINVAL, "rb_push: eps < 0");
  RBP_REQUIRE(ring->arena_off && ring->length && ring->reward && ring->advantage &&
                  ring->version && ring->arena_tokens && ring->arena_old_logp,
              RBP_EINVAL, "rb_push: null ring array");
  RBP_REQUIRE(group_off && length && src_off && reward && tokens && old_logp, RBP_EINVAL,
              "rb_push: null input array");
  RBP_REQUIRE(ring->replay_hist == nullptr ||
                  (ring->use_count != nullptr && ring->replay_bins >= 1 &&
                   ring->replay_bins <= kHistMaxBins),
              RBP_EINVAL, "rb_push: replay_hist needs use_count and 1 <= replay_bins <= %d",
              kHistMaxBins);
  hipStream_t s = rbp::as_stream(stream);
  // the first free row: just past the newest record
  int64_t base = ring->head + ring->n_live;
  if (base >= cap) base -= cap;
  // new records from index cap - n_live on overwrite live ones
  const int64_t first_evict = cap - ring->n_live;
  if (ring->replay_hist != nullptr && first_evict < n_new)
    hipLaunchKernelGGL(push_evict_kernel, dim3(rbp::ceil_div(n_new - first_evict, 256)),
                       dim3(256), 0, s, n_new, first_evict, base, cap, ring->use_count,
                       ring->replay_bins, ring->replay_hist);
  hipLaunchKernelGGL(push_rows_kernel, dim3(rbp::ceil_div(n_new, 256)), dim3(256), 0, s, n_new,
                     base, cap, ring->slot_tokens, length, reward, version, ring->arena_off,
                     ring->length, ring->reward, ring->version, ring->use_count,
                     ring->last_step);
  hipLaunchKernelGGL(push_advantage_kernel, dim3(rbp::ceil_div(n_groups, 64)), dim3(64), 0, s,
                     reward, group_off, n_groups, ddof, eps, base, cap, ring->advantage);
  int64_t by = rbp::ceil_div(ring->slot_tokens, 256);
  if (by > 16) by = 16;
  hipLaunchKernelGGL(push_copy_kernel, dim3(n_new, by), dim3(256), 0, s, base, cap,
                     ring->slot_tokens, length, src_off, tokens, old_logp, ring->arena_tokens,
                     ring->arena_old_logp);
  RBP_CHECK_LAUNCH("rb_push");
  // FIFO bookkeeping (host integers): records past the capacity evict the oldest
  const int64_t total = ring->n_live + n_new;
  const int64_t evicted = total > cap ? total - cap : 0;
  ring->head = (ring->head + evicted) % cap;
  ring->n_live = total - evicted;
  return RBP_OK;
}

extern "C" int rb_note_use(const int32_t* idx, int64_t n_draw, int64_t head, int64_t capacity,
                           int64_t step, int32_t* use_count, int64_t* last_step, int32_t* since,
                           void* ws, size_t ws_bytes, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(n_draw >= 0, RBP_EINVAL, "rb_note_use: n_draw < 0");
  RBP_REQUIRE(capacity >= 1 && capacity <= INT32_MAX && head >= 0 && head < capacity,
              RBP_EINVAL, "rb_note_use: need 1 <= capacity < 2^31 and 0 <= head < capacity");
  RBP_REQUIRE(step >= 0, RBP_EINVAL, "rb_note_use: step < 0");
  if (n_draw == 0) return RBP_OK;
  RBP_REQUIRE(idx && use_count && last_step, RBP_EINVAL, "rb_note_use: null pointer");
  const size_t need = rbp::note_use_ws(capacity);
  RBP_REQUIRE(ws && ws_bytes >= need, RBP_EWORKSPACE,
              "rb_note_use: workspace needs %zu bytes, got %zu", need, ws_bytes);
  hipStream_t s = rbp::as_stream(stream);
  int32_t* first = static_cast<int32_t*>(ws);
  int64_t blocks = rbp::ceil_div(n_draw, 256);
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(use_reset_kernel, dim3(blocks), dim3(256), 0, s, idx, n_draw, head,
                     capacity, first);
  hipLaunchKernelGGL(use_first_kernel, dim3(blocks), dim3(256), 0, s, idx, n_draw, head,
                     capacity, first);
  if (since != nullptr)
    hipLaunchKernelGGL(use_since_kernel, dim3(blocks), dim3(256), 0, s, idx, n_draw, head,
                       capacity, step, first, last_step, since);
  hipLaunchKernelGGL(use_update_kernel, dim3(blocks), dim3(256), 0, s, idx, n_draw, head,
                     capacity, step, first, use_count, last_step);
  RBP_CHECK_LAUNCH("rb_note_use");
  return RBP_OK;
}

extern "C" int rb_hist_accumulate(const int32_t* values, int64_t n, int32_t lo, int32_t n_bins,
                                  int64_t* hist, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(n >= 0, RBP_EINVAL, "rb_hist_accumulate: n < 0");
  RBP_REQUIRE(n_bins >= 1 && n_bins <= kHistMaxBins, RBP_EINVAL,
              "rb_hist_accumulate: n_bins %d outside [1, %d]", n_bins, kHistMaxBins);
  if (n == 0) return RBP_OK;
  RBP_REQUIRE(values && hist, RBP_EINVAL, "rb_hist_accumulate: null pointer");
  int64_t blocks = rbp::ceil_div(n, 256 * 8);
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(hist_kernel, dim3(blocks), dim3(256), 0, rbp::as_stream(stream), values, n,
                     lo, n_bins, hist);
  RBP_CHECK_LAUNCH("rb_hist_accumulate");
  return RBP_OK;
}
