// Policy log-probabilities of replayed tokens and their backward
// (policy_logprob_fwd, policy_logprob_bwd).
//
// Paper: App. D.2 -- the GRPO ratio needs pi_theta of every replayed token
// under the current policy; temperature 1, untied LM head.  With z_t = W h_t:
//   lse_t = log sum_v exp(z_{t,v}),  logp_t = z_{t,y_t} - lse_t,
//   dz_t = dlogp_t (e_{y_t} - softmax(z_t)),  dh_t = W^T dz_t,  dW = sum_t dz_t h_t^T.
//
// Forward: one bf16 MFMA product Z^T = W H^T per 256 (vocab) x 256 (token)
// tile; the tile never leaves registers -- its epilogue reduces each token
// column to a (max, sum exp) pair over the tile's 256 vocabulary rows, written
// as a partial.  A merge pass combines a token's partials into lse and forms
// the target logit z_{t,y_t} = h_t . W_{y_t} directly (one dot product).
//
// Backward, per chunk of Tc tokens:
//   1. the same product is recomputed; its epilogue turns the tile into
//      dz = dlogp (onehot - exp(z - lse)), rounded to bf16, into a [Tc, Vp]
//      workspace (Vp = V rounded up to 256; padding written as zeros);
//   2. dH^T = W^T dz^T  (A = W read vocab-major, transposed in the loader);
//   3. dW^T = H^T dz    (both operands token-major, transposed in the loader).
// All three are MFMA-bound; no floating-point atomics are used, so results are
// bitwise reproducible.

#include <cmath>

#include "gemm_core.h"
#include "gemm_dma.h"
#include "rbp_internal.h"

namespace {

using rbp::gemm::acc_m;
using rbp::gemm::acc_n;
using rbp::gemm::f32x16;
using rbp::gemm::kLdsBytes;
using rbp::gemm::mainloop;
using rbp::gemm::mainloop_dma;
using rbp::gemm::map_tile;
using rbp::gemm::Operand;

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kGroupLogits = 4;
constexpr int kGroupGrad = 4;

#define RBP_GEMM_KERNEL \
  __global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1)))

// Logit products (K-major operands, direct HBM -> LDS loads): 8 waves, two per
// SIMD, so that enough waves keep loads in flight to feed 256 x 256 tiles.
using GL = rbp::gemm::Grid8;
#define RBP_LOGITS_KERNEL                                                        \
  __global__ __attribute__((amdgpu_flat_work_group_size(GL::kThreads, GL::kThreads), \
                            amdgpu_waves_per_eu(GL::kWaves / 4, GL::kWaves / 4)))

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// Forward tile: partial (max, sum exp) of each token column over 256 vocab rows.
RBP_LOGITS_KERNEL void logits_lse_partial_kernel(const uint16_t* __restrict__ W,
                                                 const uint16_t* __restrict__ H, int64_t T,
                                                 int32_t d, int32_t V, int64_t tiles_m,
                                                 int64_t tiles_n, float2* __restrict__ part,
                                                 int64_t ld_part) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  int64_t tm, tn;
  map_tile(blockIdx.x, tiles_m, tiles_n, kGroupLogits, tm, tn);
  const int64_t m0 = tm * 256, n0 = tn * 256;
  const Operand A{W, d, V, d};
  const Operand B{H, d, T, d};
  f32x16 acc[GL::MI][GL::NI];
  mainloop_dma<GL>(A, B, m0, n0, 0, d, smem, acc);

  float2* lds_ms = reinterpret_cast<float2*>(smem);  // [wm][256 columns]
  const int lane = threadIdx.x & 63;
  const int64_t vlim = (int64_t)V - m0;
#pragma unroll
  for (int ni = 0; ni < GL::NI; ++ni) {
    float mx = -INFINITY;
#pragma unroll
    for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        if (GL::row(mi, r) < vlim) mx = fmaxf(mx, acc[mi][ni][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float sum = 0.0f;
    if (mx != -INFINITY) {
      const float mb = mx * kLog2e;
#pragma unroll
      for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (GL::row(mi, r) < vlim) sum += exp2f(fmaf(acc[mi][ni][r], kLog2e, -mb));
    }
    sum += __shfl_xor(sum, 32, 64);
    if (lane < 32) lds_ms[GL::wm() * 256 + GL::col(ni)] = make_float2(mx, sum);
  }
  __syncthreads();
  if (threadIdx.x < 256) {
    const int col = threadIdx.x;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < GL::WM; ++w) M = fmaxf(M, lds_ms[w * 256 + col].x);
    float S = 0.0f;
#pragma unroll
    for (int w = 0; w < GL::WM; ++w) {
      const float2 q = lds_ms[w * 256 + col];
      if (q.x != -INFINITY) S += q.y * exp2f((q.x - M) * kLog2e);
    }
    const int64_t t = n0 + col;
    if (t < T) part[t * ld_part + tm] = make_float2(M, S);
  }
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// One wave per token: merge the partials into lse, dot h_t . W_{y_t}.
__global__ void __launch_bounds__(256) lse_merge_kernel(
    const float2* __restrict__ part, int64_t ld_part, int64_t n_part,
    const uint16_t* __restrict__ H, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ seq, int64_t T, int32_t d,
    int32_t V, float* __restrict__ logp, float* __restrict__ lse) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T) return;
  if (seq != nullptr && seq[t] < 0) {
    if (lane == 0) {
      logp[t] = 0.0f;
      lse[t] = 0.0f;
    }
    return;
  }
  const float2* p = part + t * ld_part;
  float M = -INFINITY;
  for (int64_t i = lane; i < n_part; i += 64) M = fmaxf(M, p[i].x);
  M = wave_max(M);
  float S = 0.0f;
  for (int64_t i = lane; i < n_part; i += 64) {
    const float2 q = p[i];
    S += q.y * exp2f((q.x - M) * kLog2e);
  }
  S = wave_sum(S);
  const int32_t y = tokens[t];
  const bool y_ok = y >= 0 && y < V;
  const uint16_t* h = H + t * d;
  const uint16_t* w = W + (int64_t)(y_ok ? y : 0) * d;
  float z = 0.0f;
  for (int c = lane; c < d / 8; c += 64) {
    const uint4 hv = *reinterpret_cast<const uint4*>(h + c * 8);
    const uint4 wv = *reinterpret_cast<const uint4*>(w + c * 8);
    const uint32_t hh[4] = {hv.x, hv.y, hv.z, hv.w}, ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      z = fmaf(bf16_to_f32((uint16_t)(hh[q] & 0xffff)), bf16_to_f32((uint16_t)(ww[q] & 0xffff)), z);
      z = fmaf(bf16_to_f32((uint16_t)(hh[q] >> 16)), bf16_to_f32((uint16_t)(ww[q] >> 16)), z);
    }
  }
  z = wave_sum(z);
  if (lane == 0) {
    const float l = M + logf(S);
    lse[t] = l;
    logp[t] = y_ok ? z - l : NAN;
  }
}

// Backward step 1: recompute the tile, write dz = dlogp (onehot - p) as bf16.
RBP_LOGITS_KERNEL void grad_logits_kernel(const uint16_t* __restrict__ W,
                                          const uint16_t* __restrict__ Hc, int64_t Tn,
                                          int32_t d, int32_t V, const int32_t* __restrict__ tokens,
                                          const int32_t* __restrict__ seq,
                                          const float* __restrict__ lse,
                                          const float* __restrict__ dlogp,
                                          uint16_t* __restrict__ G, int64_t ldG, int64_t tiles_m,
                                          int64_t tiles_n) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  int64_t tm, tn;
  map_tile(blockIdx.x, tiles_m, tiles_n, kGroupLogits, tm, tn);
  const int64_t m0 = tm * 256, n0 = tn * 256;
  const Operand A{W, d, V, d};
  const Operand B{Hc, d, Tn, d};
  f32x16 acc[GL::MI][GL::NI];
  mainloop_dma<GL>(A, B, m0, n0, 0, d, smem, acc);

  const int64_t vlim = (int64_t)V - m0;
#pragma unroll
  for (int ni = 0; ni < GL::NI; ++ni) {
    const int64_t t = n0 + GL::col(ni);
    float ls = 0.0f, dl = 0.0f;
    int64_t y = -1;
    if (t < Tn && (seq == nullptr || seq[t] >= 0)) {
      ls = lse[t];
      dl = dlogp[t];
      y = (int64_t)tokens[t] - m0;  // target row within this tile
    }
    const float lsb = ls * kLog2e;
    uint16_t* grow = G + t * ldG + m0;
#pragma unroll
    for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        float g[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int v = GL::row(mi, rg * 4 + i);
          const float p = exp2f(fmaf(acc[mi][ni][rg * 4 + i], kLog2e, -lsb));
          const float oh = (v == y) ? 1.0f : 0.0f;
          g[i] = (v < vlim) ? dl * (oh - p) : 0.0f;
        }
        uint2 pk;
        pk.x = pack_bf16x2(g[0], g[1]);
        pk.y = pack_bf16x2(g[2], g[3]);
        *reinterpret_cast<uint2*>(grow + GL::row(mi, rg * 4)) = pk;
      }
  }
}

// Backward step 2: dH[t][m] = sum_v W[v][m] dz[t][v].
RBP_GEMM_KERNEL void dhidden_kernel(const uint16_t* __restrict__ W,
                                    const uint16_t* __restrict__ G, int64_t Tn, int32_t d,
                                    int32_t V, int64_t ldG, float* __restrict__ dH,
                                    int64_t tiles_m, int64_t tiles_n) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  int64_t tm, tn;
  map_tile(blockIdx.x, tiles_m, tiles_n, kGroupGrad, tm, tn);
  const int64_t m0 = tm * 256, n0 = tn * 256;
  const Operand A{W, d, d, V};      // (m = hidden unit, k = vocab): W[k * d + m]
  const Operand B{G, ldG, Tn, ldG}; // (n = token, k = vocab): G[n * ldG + k]
  f32x16 acc[4][4];
  mainloop<false, true>(A, B, m0, n0, 0, ldG, smem, acc);
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
    const int64_t t = n0 + acc_n(ni);
    if (t >= Tn) continue;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int64_t m = m0 + acc_m(mi, rg * 4);
        if (m < d) {
          float4 v = make_float4(acc[mi][ni][rg * 4 + 0], acc[mi][ni][rg * 4 + 1],
                                 acc[mi][ni][rg * 4 + 2], acc[mi][ni][rg * 4 + 3]);
          *reinterpret_cast<float4*>(dH + t * d + m) = v;
        }
      }
  }
}

// Backward step 3: dW[v][m] (+)= sum_t H[t][m] dz[t][v].
RBP_GEMM_KERNEL void dweight_kernel(const uint16_t* __restrict__ Hc,
                                    const uint16_t* __restrict__ G, int64_t Tn, int32_t d,
                                    int32_t V, int64_t ldG, float* __restrict__ dW,
                                    int accumulate, int64_t tiles_m, int64_t tiles_n) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  int64_t tm, tn;
  map_tile(blockIdx.x, tiles_m, tiles_n, kGroupGrad, tm, tn);
  const int64_t m0 = tm * 256, n0 = tn * 256;
  const Operand A{Hc, d, d, Tn};     // (m = hidden unit, k = token): H[k * d + m]
  const Operand B{G, ldG, ldG, Tn};  // (n = vocab, k = token): G[k * ldG + n]
  f32x16 acc[4][4];
  mainloop<false, false>(A, B, m0, n0, 0, Tn, smem, acc);
#pragma unroll
  for (int ni = 0; ni < 4; ++ni) {
    const int64_t v = n0 + acc_n(ni);
    if (v >= V) continue;
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int64_t m = m0 + acc_m(mi, rg * 4);
        if (m < d) {
          float4* dst = reinterpret_cast<float4*>(dW + v * d + m);
          float4 val = make_float4(acc[mi][ni][rg * 4 + 0], acc[mi][ni][rg * 4 + 1],
                                   acc[mi][ni][rg * 4 + 2], acc[mi][ni][rg * 4 + 3]);
          if (accumulate) {
            const float4 o = *dst;
            val.x += o.x;
            val.y += o.y;
            val.z += o.z;
            val.w += o.w;
          }
          *dst = val;
        }
      }
  }
}

__global__ void __launch_bounds__(256) fill_zero_kernel(float* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = 0.0f;
}

int64_t round256(int64_t x) { return (x + 255) / 256 * 256; }

}  // namespace

size_t rbp::logprob_fwd_ws(int64_t T, int32_t V) {
  const int64_t n_part = ceil_div(V, 256);
  return align_up(sizeof(float2) * (size_t)(T < 1 ? 1 : T) * (size_t)n_part, 256);
}

size_t rbp::logprob_bwd_ws(int64_t Tc, int32_t /*d*/, int32_t V) {
  return align_up(sizeof(uint16_t) * (size_t)round256(Tc < 1 ? 1 : Tc) * (size_t)round256(V),
                  256);
}

extern "C" int policy_logprob_fwd(const uint16_t* hidden, const uint16_t* W,
                                  const int32_t* tokens, const int32_t* seq_of_token, int64_t T,
                                  int32_t d, int32_t V, float* logp, float* lse, void* ws,
                                  size_t ws_bytes, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(T >= 0 && d >= 1 && V >= 1, RBP_EINVAL,
              "policy_logprob_fwd: need T >= 0, d >= 1, V >= 1");
  RBP_REQUIRE(d % 8 == 0, RBP_EUNSUPPORTED, "policy_logprob_fwd: d %% 8 != 0 (d = %d)", d);
  if (T == 0) return RBP_OK;
  RBP_REQUIRE(hidden && W && tokens && logp && lse, RBP_EINVAL,
              "policy_logprob_fwd: null pointer");
  const size_t need = rbp::logprob_fwd_ws(T, V);
  RBP_REQUIRE(ws && ws_bytes >= need, RBP_EWORKSPACE,
              "policy_logprob_fwd: workspace needs %zu bytes, got %zu", need, ws_bytes);
  hipStream_t s = rbp::as_stream(stream);
  const int64_t tiles_m = rbp::ceil_div(V, 256), tiles_n = rbp::ceil_div(T, 256);
  float2* part = static_cast<float2*>(ws);
  hipLaunchKernelGGL(logits_lse_partial_kernel, dim3(tiles_m * tiles_n), dim3(GL::kThreads), 0, s, W,
                     hidden, T, d, V, tiles_m, tiles_n, part, tiles_m);
  hipLaunchKernelGGL(lse_merge_kernel, dim3(rbp::ceil_div(T, 4)), dim3(256), 0, s, part, tiles_m,
                     tiles_m, hidden, W, tokens, seq_of_token, T, d, V, logp, lse);
  RBP_CHECK_LAUNCH("policy_logprob_fwd");
  return RBP_OK;
}

extern "C" int policy_logprob_bwd(const uint16_t* hidden, const uint16_t* W,
                                  const int32_t* tokens, const int32_t* seq_of_token,
                                  const float* lse, const float* dlogp, int64_t T, int32_t d,
                                  int32_t V, float* dhidden, float* dW, int accumulate_dW,
                                  void* ws, size_t ws_bytes, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(T >= 0 && d >= 1 && V >= 1, RBP_EINVAL,
              "policy_logprob_bwd: need T >= 0, d >= 1, V >= 1");
  RBP_REQUIRE(d % 8 == 0, RBP_EUNSUPPORTED, "policy_logprob_bwd: d %% 8 != 0 (d = %d)", d);
  RBP_REQUIRE(W && dW, RBP_EINVAL, "policy_logprob_bwd: null pointer");
  RBP_REQUIRE(T == 0 || (hidden && tokens && lse && dlogp && dhidden), RBP_EINVAL,
              "policy_logprob_bwd: null pointer");
  hipStream_t s = rbp::as_stream(stream);
  const int64_t Vp = round256(V);
  const int64_t tiles_d = rbp::ceil_div(d, 256), tiles_v = Vp / 256;
  if (T == 0) {
    if (!accumulate_dW) {
      const int64_t n = (int64_t)V * d;
      int64_t blocks = rbp::ceil_div(n, 256);
      if (blocks > 65536) blocks = 65536;
      hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, s, dW, n);
      RBP_CHECK_LAUNCH("policy_logprob_bwd");
    }
    return RBP_OK;
  }
  // largest chunk (multiple of 256 tokens) whose dz workspace fits
  int64_t Tc = ws ? (int64_t)(ws_bytes / (sizeof(uint16_t) * (size_t)Vp)) / 256 * 256 : 0;
  if (Tc > round256(T)) Tc = round256(T);
  RBP_REQUIRE(Tc >= 256, RBP_EWORKSPACE,
              "policy_logprob_bwd: workspace of %zu bytes holds no 256-token chunk (needs %zu)",
              ws_bytes, rbp::logprob_bwd_ws(256, d, V));
  uint16_t* G = static_cast<uint16_t*>(ws);
  for (int64_t t0 = 0; t0 < T; t0 += Tc) {
    const int64_t Tn = (T - t0) < Tc ? (T - t0) : Tc;
    const int64_t tiles_t = rbp::ceil_div(Tn, 256);
    const uint16_t* Hc = hidden + t0 * d;
    hipLaunchKernelGGL(grad_logits_kernel, dim3(tiles_v * tiles_t), dim3(GL::kThreads), 0, s, W, Hc, Tn,
                       d, V, tokens + t0, seq_of_token ? seq_of_token + t0 : nullptr, lse + t0,
                       dlogp + t0, G, Vp, tiles_v, tiles_t);
    hipLaunchKernelGGL(dhidden_kernel, dim3(tiles_d * tiles_t), dim3(256), 0, s, W, G, Tn, d, V,
                       Vp, dhidden + t0 * d, tiles_d, tiles_t);
    hipLaunchKernelGGL(dweight_kernel, dim3(tiles_d * tiles_v), dim3(256), 0, s, Hc, G, Tn, d, V,
                       Vp, dW, (accumulate_dW || t0 > 0) ? 1 : 0, tiles_d, tiles_v);
  }
  RBP_CHECK_LAUNCH("policy_logprob_bwd");
  return RBP_OK;
}
