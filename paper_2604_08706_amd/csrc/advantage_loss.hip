// Group advantage at insert (rb_group_advantage) and the clipped GRPO loss
// with its gradient w.r.t. the token log-probabilities (policy_loss_fwd_bwd).
//
// Paper, App. D.2: A_i = (r_i - mean) / std over the G rollouts of a prompt,
// computed when the group is generated; the objective is the expectation of
// min(rho A, clip(rho, 1 - eps_low, 1 + eps_high) A) with old probabilities
// recorded at generation, eps = 0.2, no KL term.  Token-level ratio and
// per-sequence token means, loss = -J (see rbpolicy.h for the exact form).
//
// The loss pass is HBM/latency bound (~20 B per token).  Per-token work is a
// grid-stride loop; the five sums are reduced per block in a fixed butterfly
// order and then summed over blocks by one small block in block order, so the
// result is bitwise reproducible.

#include "rbp_internal.h"

namespace {

constexpr int kLossThreads = 256;
constexpr int kLossMaxBlocks = 1024;
constexpr int kNumSums = 5;  // -sum w*l, sum rho, n clipped, n valid, sum l

__global__ void __launch_bounds__(64) group_advantage_kernel(
    const float* __restrict__ reward, const int32_t* __restrict__ group_off,
    int32_t n_groups, int32_t ddof, float eps, float* __restrict__ adv) {
  const int32_t g = blockIdx.x * 64 + threadIdx.x;
  if (g >= n_groups) return;
  const int32_t lo = group_off[g], hi = group_off[g + 1];
  const int32_t n = hi - lo;
  if (n <= 0) return;
  float sum = 0.0f;
  for (int32_t i = lo; i < hi; ++i) sum += reward[i];
  const float mean = sum / (float)n;
  float ss = 0.0f;
  for (int32_t i = lo; i < hi; ++i) {
    const float dv = reward[i] - mean;
    ss = fmaf(dv, dv, ss);
  }
  if (ss == 0.0f || n - ddof <= 0) {
    for (int32_t i = lo; i < hi; ++i) adv[i] = 0.0f;
    return;
  }
  const float sd = __fsqrt_rn(ss / (float)(n - ddof));
  const float denom = sd + eps;
  for (int32_t i = lo; i < hi; ++i) adv[i] = (reward[i] - mean) / denom;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__global__ void __launch_bounds__(kLossThreads) grpo_token_kernel(
    const float* __restrict__ logp, const float* __restrict__ old_logp,
    const int32_t* __restrict__ seq_of_token, const float* __restrict__ adv,
    const int32_t* __restrict__ seq_len, int64_t T, float inv_nseq, float eps_low,
    float eps_high, float* __restrict__ dlogp, float* __restrict__ partials) {
  float acc[kNumSums] = {0.f, 0.f, 0.f, 0.f, 0.f};
  const float lo_b = 1.0f - eps_low, hi_b = 1.0f + eps_high;
  for (int64_t t = (int64_t)blockIdx.x * kLossThreads + threadIdx.x; t < T;
       t += (int64_t)gridDim.x * kLossThreads) {
    const int32_t s = seq_of_token[t];
    float g = 0.0f;
    if (s >= 0) {
      const float A = adv[s];
      const float w = inv_nseq / (float)seq_len[s];
      const float rho = expf(logp[t] - old_logp[t]);
      const float clipped = fminf(fmaxf(rho, lo_b), hi_b);
      const float term = fminf(rho * A, clipped * A);
      const bool cut = (A > 0.0f && rho > hi_b) || (A < 0.0f && rho < lo_b);
      g = cut ? 0.0f : -A * rho * w;
      acc[0] -= term * w;
      acc[1] += rho;
      acc[2] += cut ? 1.0f : 0.0f;
      acc[3] += 1.0f;
      acc[4] += term;
    }
    dlogp[t] = g;
  }
  __shared__ float lds[kLossThreads / 64][kNumSums];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < kNumSums; ++k) {
    const float v = wave_sum(acc[k]);
    if (lane == 0) lds[wave][k] = v;
  }
  __syncthreads();
  if (threadIdx.x < kNumSums) {
    float v = 0.0f;
    for (int w = 0; w < kLossThreads / 64; ++w) v += lds[w][threadIdx.x];
    partials[(int64_t)blockIdx.x * kNumSums + threadIdx.x] = v;
  }
}

__global__ void __launch_bounds__(64) grpo_finalize_kernel(const float* __restrict__ partials,
                                                           int nblocks,
                                                           float* __restrict__ loss_accum,
                                                           float* __restrict__ stats) {
  // one lane per sum, blocks added in block order
  const int k = threadIdx.x;
  if (k >= kNumSums) return;
  float v = 0.0f;
  for (int b = 0; b < nblocks; ++b) v += partials[b * kNumSums + k];
  if (k == 0)
    loss_accum[0] += v;
  else
    stats[k - 1] += v;
}

}  // namespace

size_t rbp::loss_ws(int64_t /*T*/) {
  return align_up(sizeof(float) * kLossMaxBlocks * kNumSums, 256);
}

extern "C" int rb_group_advantage(const float* reward, const int32_t* group_off,
                                  int32_t n_groups, int32_t ddof, float eps, float* adv,
                                  void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(reward && group_off && adv, RBP_EINVAL, "rb_group_advantage: null pointer");
  RBP_REQUIRE(n_groups >= 0, RBP_EINVAL, "rb_group_advantage: n_groups < 0");
  RBP_REQUIRE(ddof == 0 || ddof == 1, RBP_EINVAL, "rb_group_advantage: ddof must be 0 or 1");
  RBP_REQUIRE(eps >= 0.0f, RBP_EINVAL, "rb_group_advantage: eps < 0");
  if (n_groups == 0) return RBP_OK;
  hipLaunchKernelGGL(group_advantage_kernel, dim3((n_groups + 63) / 64), dim3(64), 0,
                     rbp::as_stream(stream), reward, group_off, n_groups, ddof, eps, adv);
  RBP_CHECK_LAUNCH("rb_group_advantage");
  return RBP_OK;
}

extern "C" int policy_loss_fwd_bwd(const float* logp, const float* old_logp,
                                   const int32_t* seq_of_token, const float* adv,
                                   const int32_t* seq_len, int64_t T, int32_t B,
                                   int64_t n_seq_total, float eps_low, float eps_high,
                                   float* loss_accum, float* dlogp, float* stats, void* ws,
                                   size_t ws_bytes, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(T >= 0, RBP_EINVAL, "policy_loss_fwd_bwd: T < 0");
  RBP_REQUIRE(B >= 1 && n_seq_total >= 1, RBP_EINVAL,
              "policy_loss_fwd_bwd: need B >= 1 and n_seq_total >= 1");
  RBP_REQUIRE(eps_low >= 0.0f && eps_high >= 0.0f, RBP_EINVAL,
              "policy_loss_fwd_bwd: negative clip range");
  RBP_REQUIRE(adv && seq_len && loss_accum && stats, RBP_EINVAL,
              "policy_loss_fwd_bwd: null pointer");
  RBP_REQUIRE(T == 0 || (logp && old_logp && seq_of_token && dlogp), RBP_EINVAL,
              "policy_loss_fwd_bwd: null per-token pointer");
  const size_t need = rbp::loss_ws(T);
  RBP_REQUIRE(ws && ws_bytes >= need, RBP_EWORKSPACE,
              "policy_loss_fwd_bwd: workspace needs %zu bytes, got %zu", need, ws_bytes);
  hipStream_t s = rbp::as_stream(stream);
  int64_t nb = rbp::ceil_div(T, kLossThreads * 4);
  if (nb < 1) nb = 1;
  if (nb > kLossMaxBlocks) nb = kLossMaxBlocks;
  float* partials = static_cast<float*>(ws);
  const float inv_nseq = (float)(1.0 / (double)n_seq_total);
  hipLaunchKernelGGL(grpo_token_kernel, dim3(nb), dim3(kLossThreads), 0, s, logp, old_logp,
                     seq_of_token, adv, seq_len, T, inv_nseq, eps_low, eps_high, dlogp,
                     partials);
  hipLaunchKernelGGL(grpo_finalize_kernel, dim3(1), dim3(64), 0, s, partials, (int)nb,
                     loss_accum, stats);
  RBP_CHECK_LAUNCH("policy_loss_fwd_bwd");
  return RBP_OK;
}
