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

#include "group_advantage.h"
#include "rbp_internal.h"

namespace {

constexpr int kLossThreads = 256;
constexpr int kLossMaxBlocks = 1024;
constexpr int kNumSums = 5;  // -sum w*l, sum rho, n clipped, n valid, sum l

constexpr int kAdvGroups = 256;   // groups per block, one thread each
constexpr int kAdvStage = 4096;   // records a block stages through LDS

// Block b takes groups [256 b, 256 b + 256), whose records form one
// contiguous range.  When that range fits the stage, it is read into LDS and
// the advantages written back with coalesced accesses (a thread per group
// reading its own records from HBM makes a wave's loads 4 G bytes apart);
// longer ranges take the direct path.  Same arithmetic either way.
__global__ void __launch_bounds__(kAdvGroups) group_advantage_kernel(
    const float* __restrict__ reward, const int32_t* __restrict__ group_off,
    int32_t n_groups, int32_t ddof, float eps, float* __restrict__ adv) {
  __shared__ float r_s[kAdvStage], a_s[kAdvStage];
  const int32_t g0 = blockIdx.x * kAdvGroups;
  const int32_t g1 = g0 + kAdvGroups < n_groups ? g0 + kAdvGroups : n_groups;
  const int32_t g = g0 + threadIdx.x;
  const int32_t lo = group_off[g0], n = group_off[g1] - lo;
  if (n > kAdvStage) {
    if (g < g1)
      rbp::group_advantage(reward, group_off[g], group_off[g + 1], ddof, eps,
                           [&](int32_t i, float a) { adv[i] = a; });
    return;
  }
  for (int32_t k = threadIdx.x; k < n; k += kAdvGroups) r_s[k] = reward[lo + k];
  __syncthreads();
  if (g < g1)
    rbp::group_advantage(r_s, group_off[g] - lo, group_off[g + 1] - lo, ddof, eps,
                         [&](int32_t i, float a) { a_s[i] = a; });
  __syncthreads();
  for (int32_t k = threadIdx.x; k < n; k += kAdvGroups) adv[lo + k] = a_s[k];
}

constexpr int kSeqThreads = 256;  // threads per sequence of the whole-sequence ratio

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

// ---- objective variants -------------------------------------------------

__global__ void __launch_bounds__(64) asymre_coef_kernel(const float* __restrict__ reward,
                                                         const int32_t* __restrict__ group_off,
                                                         int32_t n_groups, float delta_v,
                                                         float* __restrict__ coef) {
  const int32_t g = blockIdx.x * 64 + threadIdx.x;
  if (g >= n_groups) return;
  const int32_t lo = group_off[g], hi = group_off[g + 1];
  if (hi <= lo) return;
  // fp64 as in the group advantage: the group mean of fp32 rewards is exact,
  // so equal rewards give coef = -delta_v exactly; one rounding at the end.
  double sum = 0.0;
  for (int32_t i = lo; i < hi; ++i) sum += (double)reward[i];
  const double base = sum / (double)(hi - lo) + (double)delta_v;
  for (int32_t i = lo; i < hi; ++i) coef[i] = (float)((double)reward[i] - base);
}

// AsymRE per token: dlogp = -c / n_seq; sums {-sum c logp / n_seq, valid, sum c logp}
// in the slots {0, 3, 4} of the shared partial layout (1, 2 unused).
__global__ void __launch_bounds__(kLossThreads) asymre_token_kernel(
    const float* __restrict__ logp, const int32_t* __restrict__ seq_of_token,
    const float* __restrict__ coef, int64_t T, float inv_nseq, float* __restrict__ dlogp,
    float* __restrict__ partials) {
  float s_cl = 0.0f, n_valid = 0.0f;
  for (int64_t t = (int64_t)blockIdx.x * kLossThreads + threadIdx.x; t < T;
       t += (int64_t)gridDim.x * kLossThreads) {
    const int32_t s = seq_of_token[t];
    float g = 0.0f;
    if (s >= 0) {
      const float c = coef[s];
      g = -c * inv_nseq;
      s_cl = fmaf(c, logp[t], s_cl);
      n_valid += 1.0f;
    }
    dlogp[t] = g;
  }
  __shared__ float lds[kLossThreads / 64][2];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float a = wave_sum(s_cl), b = wave_sum(n_valid);
  if (lane == 0) {
    lds[wave][0] = a;
    lds[wave][1] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float v0 = 0.0f, v1 = 0.0f;
    for (int w = 0; w < kLossThreads / 64; ++w) {
      v0 += lds[w][0];
      v1 += lds[w][1];
    }
    float* p = partials + (int64_t)blockIdx.x * kNumSums;
    p[0] = -v0 * inv_nseq;
    p[1] = 0.0f;
    p[2] = 0.0f;
    p[3] = v1;
    p[4] = v0;
  }
}

// Sum k of the partials over blocks (one wave per sum, fixed order), added to
// out[k]; AsymRE and the sequence form share the partial layout above.
__global__ void __launch_bounds__(64) sums_finalize_kernel(const float* __restrict__ partials,
                                                           int nblocks, int k_first, int k_count,
                                                           float* __restrict__ loss_accum,
                                                           float* __restrict__ stats) {
  const int lane = threadIdx.x & 63;
  const int k = blockIdx.x;
  float v = 0.0f;
  for (int b = lane; b < nblocks; b += 64) v += partials[b * kNumSums + k];
  v = wave_sum(v);
  if (lane == 0) {
    if (k == 0)
      loss_accum[0] += v;
    else if (k >= k_first && k < k_first + k_count)
      stats[k - k_first] += v;
  }
}

// Whole-sequence ratio: one block per sequence sums log-ratios over its
// tokens (thread-strided, fixed butterfly per wave, the four wave sums in
// order), forms rho_i, the term and the gradient, writes dlogp over the
// sequence and the per-sequence values into `seqv` ([B][4]: -l_i / n_seq,
// rho_i, clipped, l_i).
__global__ void __launch_bounds__(kSeqThreads) seq_ratio_kernel(
    const float* __restrict__ logp, const float* __restrict__ old_logp,
    const int32_t* __restrict__ cu, const float* __restrict__ adv, float inv_nseq,
    float eps_low, float eps_high, float* __restrict__ dlogp, float* __restrict__ seqv) {
  __shared__ float red[kSeqThreads / 64];
  const int32_t i = blockIdx.x;
  const int lane = threadIdx.x & 63;
  const int64_t lo = cu[i], hi = cu[i + 1];
  float s = 0.0f;
  for (int64_t t = lo + threadIdx.x; t < hi; t += kSeqThreads) s += logp[t] - old_logp[t];
  s = wave_sum(s);
  if (lane == 0) red[threadIdx.x >> 6] = s;
  __syncthreads();
  s = red[0];
#pragma unroll
  for (int w = 1; w < kSeqThreads / 64; ++w) s += red[w];
  const float rho = expf(s);
  const float A = adv[i];
  const float lo_b = 1.0f - eps_low, hi_b = 1.0f + eps_high;
  const float term = fminf(rho * A, fminf(fmaxf(rho, lo_b), hi_b) * A);
  const bool cut = (A > 0.0f && rho > hi_b) || (A < 0.0f && rho < lo_b);
  const float g = cut ? 0.0f : -A * rho * inv_nseq;
  for (int64_t t = lo + threadIdx.x; t < hi; t += kSeqThreads) dlogp[t] = g;
  if (threadIdx.x == 0) {
    float* v = seqv + (int64_t)i * 4;
    v[0] = -term * inv_nseq;
    v[1] = rho;
    v[2] = cut ? 1.0f : 0.0f;
    v[3] = term;
  }
}

// Partials of the per-sequence values: block b covers sequences
// [b * 256, b * 256 + 256), in the shared layout {-sum l/n, sum rho, clipped,
// sequences, sum l}.
__global__ void __launch_bounds__(256) seq_partials_kernel(const float* __restrict__ seqv,
                                                           int32_t B,
                                                           float* __restrict__ partials) {
  const int32_t i = blockIdx.x * 256 + threadIdx.x;
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  float n = 0.0f;
  if (i < B) {
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = seqv[(int64_t)i * 4 + k];
    n = 1.0f;
  }
  __shared__ float lds[4][kNumSums];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const float r[kNumSums] = {wave_sum(v[0]), wave_sum(v[1]), wave_sum(v[2]), wave_sum(n),
                             wave_sum(v[3])};
  if (lane == 0) {
#pragma unroll
    for (int k = 0; k < kNumSums; ++k) lds[wave][k] = r[k];
  }
  __syncthreads();
  if (threadIdx.x < kNumSums) {
    float a = 0.0f;
    for (int w = 0; w < 4; ++w) a += lds[w][threadIdx.x];
    partials[(int64_t)blockIdx.x * kNumSums + threadIdx.x] = a;
  }
}

// dlogp = 0 for tokens [cu[B], T), past the last sequence.
__global__ void __launch_bounds__(256) zero_tail_kernel(const int32_t* __restrict__ cu, int32_t B,
                                                        int64_t T, float* __restrict__ dlogp) {
  const int64_t start = cu[B];
  for (int64_t t = start + (int64_t)blockIdx.x * 256 + threadIdx.x; t < T;
       t += (int64_t)gridDim.x * 256)
    dlogp[t] = 0.0f;
}

}  // namespace

size_t rbp::loss_ws(int64_t /*T*/) {
  return align_up(sizeof(float) * kLossMaxBlocks * kNumSums, 256);
}

size_t rbp::loss_seq_ws(int64_t B) {
  // per-sequence values [B][4], then one partial row per 256 sequences
  const int64_t n = B < 1 ? 1 : B;
  return align_up(sizeof(float) * (size_t)n * 4, 256) +
         align_up(sizeof(float) * (size_t)ceil_div(n, 256) * kNumSums, 256);
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
  hipLaunchKernelGGL(group_advantage_kernel, dim3(rbp::ceil_div(n_groups, kAdvGroups)),
                     dim3(kAdvGroups), 0, rbp::as_stream(stream), reward, group_off, n_groups,
                     ddof, eps, adv);
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

extern "C" int rb_asymre_coef(const float* reward, const int32_t* group_off, int32_t n_groups,
                              float delta_v, float* coef, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(n_groups >= 0, RBP_EINVAL, "rb_asymre_coef: n_groups < 0");
  if (n_groups == 0) return RBP_OK;
  RBP_REQUIRE(reward && group_off && coef, RBP_EINVAL, "rb_asymre_coef: null pointer");
  hipLaunchKernelGGL(asymre_coef_kernel, dim3((n_groups + 63) / 64), dim3(64), 0,
                     rbp::as_stream(stream), reward, group_off, n_groups, delta_v, coef);
  RBP_CHECK_LAUNCH("rb_asymre_coef");
  return RBP_OK;
}

extern "C" int policy_asymre_fwd_bwd(const float* logp, const int32_t* seq_of_token,
                                     const float* coef, int64_t T, int32_t B, int64_t n_seq_total,
                                     float* loss_accum, float* dlogp, float* stats, void* ws,
                                     size_t ws_bytes, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(T >= 0, RBP_EINVAL, "policy_asymre_fwd_bwd: T < 0");
  RBP_REQUIRE(B >= 1 && n_seq_total >= 1, RBP_EINVAL,
              "policy_asymre_fwd_bwd: need B >= 1 and n_seq_total >= 1");
  RBP_REQUIRE(coef && loss_accum && stats, RBP_EINVAL, "policy_asymre_fwd_bwd: null pointer");
  RBP_REQUIRE(T == 0 || (logp && seq_of_token && dlogp), RBP_EINVAL,
              "policy_asymre_fwd_bwd: null per-token pointer");
  const size_t need = rbp::loss_ws(T);
  RBP_REQUIRE(ws && ws_bytes >= need, RBP_EWORKSPACE,
              "policy_asymre_fwd_bwd: workspace needs %zu bytes, got %zu", need, ws_bytes);
  hipStream_t s = rbp::as_stream(stream);
  int64_t nb = rbp::ceil_div(T, kLossThreads * 4);
  if (nb < 1) nb = 1;
  if (nb > kLossMaxBlocks) nb = kLossMaxBlocks;
  float* partials = static_cast<float*>(ws);
  const float inv_nseq = (float)(1.0 / (double)n_seq_total);
  hipLaunchKernelGGL(asymre_token_kernel, dim3(nb), dim3(kLossThreads), 0, s, logp, seq_of_token,
                     coef, T, inv_nseq, dlogp, partials);
  // loss (sum 0) and stats {valid, sum c logp} = sums 3, 4
  hipLaunchKernelGGL(sums_finalize_kernel, dim3(kNumSums), dim3(64), 0, s, partials, (int)nb, 3,
                     2, loss_accum, stats);
  RBP_CHECK_LAUNCH("policy_asymre_fwd_bwd");
  return RBP_OK;
}

extern "C" int policy_loss_seq_fwd_bwd(const float* logp, const float* old_logp,
                                       const int32_t* cu_seqlens, const float* adv, int64_t T,
                                       int32_t B, int64_t n_seq_total, float eps_low,
                                       float eps_high, float* loss_accum, float* dlogp,
                                       float* stats, void* ws, size_t ws_bytes, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(T >= 0, RBP_EINVAL, "policy_loss_seq_fwd_bwd: T < 0");
  RBP_REQUIRE(B >= 1 && n_seq_total >= 1, RBP_EINVAL,
              "policy_loss_seq_fwd_bwd: need B >= 1 and n_seq_total >= 1");
  RBP_REQUIRE(eps_low >= 0.0f && eps_high >= 0.0f, RBP_EINVAL,
              "policy_loss_seq_fwd_bwd: negative clip range");
  RBP_REQUIRE(cu_seqlens && adv && loss_accum && stats, RBP_EINVAL,
              "policy_loss_seq_fwd_bwd: null pointer");
  RBP_REQUIRE(T == 0 || (logp && old_logp && dlogp), RBP_EINVAL,
              "policy_loss_seq_fwd_bwd: null per-token pointer");
  const size_t need = rbp::loss_seq_ws(B);
  RBP_REQUIRE(ws && ws_bytes >= need, RBP_EWORKSPACE,
              "policy_loss_seq_fwd_bwd: workspace needs %zu bytes, got %zu", need, ws_bytes);
  hipStream_t s = rbp::as_stream(stream);
  rbp::WsCarver c(ws);
  float* seqv = c.take<float>((size_t)B * 4);
  const int64_t nbp = rbp::ceil_div(B, 256);
  float* partials = c.take<float>((size_t)nbp * kNumSums);
  const float inv_nseq = (float)(1.0 / (double)n_seq_total);
  hipLaunchKernelGGL(seq_ratio_kernel, dim3(B), dim3(kSeqThreads), 0, s, logp, old_logp,
                     cu_seqlens, adv, inv_nseq, eps_low, eps_high, dlogp, seqv);
  if (T > 0) {
    int64_t blocks = rbp::ceil_div(T, 256);
    if (blocks > 1024) blocks = 1024;
    hipLaunchKernelGGL(zero_tail_kernel, dim3(blocks), dim3(256), 0, s, cu_seqlens, B, T, dlogp);
  }
  hipLaunchKernelGGL(seq_partials_kernel, dim3(nbp), dim3(256), 0, s, seqv, B, partials);
  // loss (sum 0) and stats {sum rho, clipped, sequences, sum l} = sums 1..4
  hipLaunchKernelGGL(sums_finalize_kernel, dim3(kNumSums), dim3(64), 0, s, partials, (int)nbp, 1,
                     4, loss_accum, stats);
  RBP_CHECK_LAUNCH("policy_loss_seq_fwd_bwd");
  return RBP_OK;
}
