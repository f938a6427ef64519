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

// Loss terms of one token (a masked token, s < 0, contributes nothing).
struct TokenTerms {
  float g, wterm, rho, cut, valid, term;
};
__device__ __forceinline__ TokenTerms token_terms(float lp, float olp, int32_t s,
                                                  const float* __restrict__ adv,
                                                  const int32_t* __restrict__ seq_len,
                                                  float inv_nseq, float lo_b, float hi_b) {
  TokenTerms r{0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (s < 0) return r;
  const float A = adv[s];
  const float w = inv_nseq / (float)seq_len[s];
  const float rho = expf(lp - olp);
  const float clipped = fminf(fmaxf(rho, lo_b), hi_b);
  const float term = fminf(rho * A, clipped * A);
  const bool cut = (A > 0.0f && rho > hi_b) || (A < 0.0f && rho < lo_b);
  r.g = cut ? 0.0f : -A * rho * w;
  r.wterm = term * w;
  r.rho = rho;
  r.cut = cut ? 1.0f : 0.0f;
  r.valid = 1.0f;
  r.term = term;
  return r;
}

// Four consecutive tokens per thread and iteration (16-byte loads and
// stores) when the arrays are 16-byte aligned; a scalar loop takes the rest.
__global__ void __launch_bounds__(kLossThreads) grpo_token_kernel(
    const float* __restrict__ logp, const float* __restrict__ old_logp,
    const int32_t* __restrict__ seq_of_token, const float* __restrict__ adv,
    const int32_t* __restrict__ seq_len, int64_t T, int vec, float inv_nseq, float eps_low,
    float eps_high, float* __restrict__ dlogp, float* __restrict__ partials) {
  float acc[kNumSums] = {0.f, 0.f, 0.f, 0.f, 0.f};
  const float lo_b = 1.0f - eps_low, hi_b = 1.0f + eps_high;
  auto add = [&](const TokenTerms& r) {
    acc[0] -= r.wterm;
    acc[1] += r.rho;
    acc[2] += r.cut;
    acc[3] += r.valid;
    acc[4] += r.term;
  };
  const int64_t T4 = vec ? T / 4 : 0;  // vec: all four arrays 16-byte aligned
  const int64_t stride = (int64_t)gridDim.x * kLossThreads;
  for (int64_t q = (int64_t)blockIdx.x * kLossThreads + threadIdx.x; q < T4; q += stride) {
    const float4 lp = reinterpret_cast<const float4*>(logp)[q];
    const float4 ol = reinterpret_cast<const float4*>(old_logp)[q];
    const int4 sq = reinterpret_cast<const int4*>(seq_of_token)[q];
    const TokenTerms a = token_terms(lp.x, ol.x, sq.x, adv, seq_len, inv_nseq, lo_b, hi_b);
    const TokenTerms b = token_terms(lp.y, ol.y, sq.y, adv, seq_len, inv_nseq, lo_b, hi_b);
    const TokenTerms c = token_terms(lp.z, ol.z, sq.z, adv, seq_len, inv_nseq, lo_b, hi_b);
    const TokenTerms e = token_terms(lp.w, ol.w, sq.w, adv, seq_len, inv_nseq, lo_b, hi_b);
    reinterpret_cast<float4*>(dlogp)[q] = make_float4(a.g, b.g, c.g, e.g);
    add(a);
    add(b);
    add(c);
    add(e);
  }
  for (int64_t t = T4 * 4 + (int64_t)blockIdx.x * kLossThreads + threadIdx.x; t < T;
       t += stride) {
    const TokenTerms a =
        token_terms(logp[t], old_logp[t], seq_of_token[t], adv, seq_len, inv_nseq, lo_b, hi_b);
    dlogp[t] = a.g;
    add(a);
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

// Wave k sums the block partials of sum k: lane l takes blocks l, l + 64, ...
// in order, then a fixed butterfly combines the lanes (bitwise reproducible).
__global__ void __launch_bounds__(64 * kNumSums) grpo_finalize_kernel(
    const float* __restrict__ partials, int nblocks, float* __restrict__ loss_accum,
    float* __restrict__ stats) {
  const int k = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float v = 0.0f;
  for (int b = lane; b < nblocks; b += 64) v += partials[b * kNumSums + k];
  v = wave_sum(v);
  if (lane == 0) {
    if (k == 0)
      loss_accum[0] += v;
    else
      stats[k - 1] += v;
  }
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
  const int vec = ((reinterpret_cast<uintptr_t>(logp) | reinterpret_cast<uintptr_t>(old_logp) |
                    reinterpret_cast<uintptr_t>(seq_of_token) | reinterpret_cast<uintptr_t>(dlogp)) &
                   15) == 0;
  hipLaunchKernelGGL(grpo_token_kernel, dim3(nb), dim3(kLossThreads), 0, s, logp, old_logp,
                     seq_of_token, adv, seq_len, T, vec, inv_nseq, eps_low, eps_high, dlogp,
                     partials);
  hipLaunchKernelGGL(grpo_finalize_kernel, dim3(1), dim3(64 * kNumSums), 0, s, partials, (int)nb,
                     loss_accum, stats);
  RBP_CHECK_LAUNCH("policy_loss_fwd_bwd");
  return RBP_OK;
}
