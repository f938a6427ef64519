// Policy log-probabilities of replayed tokens (policy_logprob_fwd).
//
// Paper: App. D.2 -- the GRPO ratio needs pi_theta of every replayed token
// under the current policy; temperature 1, untied LM head.  With z_t = W h_t:
//   lse_t = log sum_v exp(z_{t,v}),  logp_t = z_{t,y_t} - lse_t.
//
// One bf16 MFMA product Z^T = W H^T per 256 (vocab) x 256 (token) tile, on
// the persistent direct-load stream of gemm_dma.h (one 256 x 256 workgroup
// per CU), reading W and H in place; the tile never leaves registers -- its
// epilogue reduces each token column to a (max, sum exp) pair over the tile's
// 256 vocabulary rows, written as a partial.  A merge pass combines a token's
// partials into lse and forms the target logit z_{t,y_t} = h_t . W_{y_t}
// directly (one dot product).  No floating-point atomics are used, so results
// are bitwise reproducible.

#include "logits_epilogue.h"
#include "rbp_internal.h"

namespace {

using namespace rbp::lp;
using rbp::gemm::kLdsBytes;
using rbp::gemm::Tile;
using rbp::gemm::tile_stream;
using rbp::gemm::map_tile;
using rbp::gemm::Operand;

// Forward: per 256 x 256 tile, the partial (max, sum exp) of each token
// column over the tile's 256 vocabulary rows.
RBP_LOGITS_KERNEL void logits_lse_partial_kernel(const uint16_t* __restrict__ W,
                                                 const uint16_t* __restrict__ H, int64_t T,
                                                 int32_t d, int32_t V, int64_t tiles_m,
                                                 int64_t tiles_n, float2* __restrict__ part,
                                                 int64_t ld_part) {
  // two operand stages, then the cross-wave (max, sum) exchange [WM][256]
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes + GL::WM * 256 * 8];
  float2* lds_ms = reinterpret_cast<float2*>(smem + kLdsBytes);
  const Operand A{W, d, V, d};
  const Operand B{H, d, T, d};
  const int lane = threadIdx.x & 63;
  auto tile_of = [&](int32_t vid) {
    int32_t tm, tn;
    map_tile(vid, (int32_t)tiles_m, (int32_t)tiles_n, kGroupLogits, tm, tn);
    return Tile{tm * 256, tn * 256, 0, d};
  };
  auto epi = [&](int32_t vid, f32x16 (&acc)[GL::MI][GL::NI]) {
    const Tile tile = tile_of(vid);
    const int32_t vlim = V - tile.m0;
    float mx[GL::NI], sum[GL::NI];
    if (vlim >= 256)
      column_stats<true>(acc, 0, mx, sum);
    else  // last vocabulary tile: rows past V take no part
      column_stats<false>(acc, vlim - GL::row(0, 0), mx, sum);
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni)
      if (lane < 32) lds_ms[GL::wm() * 256 + GL::col(ni)] = make_float2(mx[ni], sum[ni]);
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
        if (q.x != -INFINITY) S += q.y * exp2_hw((q.x - M) * kLog2e);
      }
      const int64_t t = tile.n0 + col;
      if (t < T) part[t * ld_part + tile.m0 / 256] = make_float2(M, S);
    }
    // lds_ms is next written in the next tile's epilogue, after at least one
    // K step (and its barrier) of that tile
  };
  tile_stream<GL, false, false>(A, B, (int32_t)(tiles_m * tiles_n), smem, tile_of, epi);
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
  const float z = dot_bf16_wave(H + t * d, W + (int64_t)(y_ok ? y : 0) * d, d, lane);
  if (lane == 0) {
    const float l = M + logf(S);
    lse[t] = l;
    logp[t] = y_ok ? z - l : NAN;
  }
}

}  // namespace

size_t rbp::logprob_fwd_ws(int64_t T, int32_t V) {
  const int64_t n_part = ceil_div(V, 256);
  return align_up(sizeof(float2) * (size_t)(T < 1 ? 1 : T) * (size_t)n_part, 256);
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
  const int64_t grid = rbp::gemm::stream_grid(tiles_m * tiles_n, device_cus());
  hipLaunchKernelGGL(logits_lse_partial_kernel, dim3(grid), dim3(GL::kThreads), 0, s, W,
                     hidden, T, d, V, tiles_m, tiles_n, part, tiles_m);
  hipLaunchKernelGGL(lse_merge_kernel, dim3(rbp::ceil_div(T, 4)), dim3(256), 0, s, part, tiles_m,
                     tiles_m, hidden, W, tokens, seq_of_token, T, d, V, logp, lse);
  RBP_CHECK_LAUNCH("policy_logprob_fwd");
  return RBP_OK;
}
