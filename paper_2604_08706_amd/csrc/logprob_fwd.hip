// Policy log-probabilities of replayed tokens (policy_logprob_fwd).
//
// Paper: App. D.2 -- the GRPO ratio needs pi_theta of every replayed token
// under the current policy; temperature 1, untied LM head.  With z_t = W h_t:
//   lse_t = log sum_v exp(z_{t,v}),  logp_t = z_{t,y_t} - lse_t.
//
// One bf16 MFMA product Z^T = W H^T per 256 (vocab) x 256 (token) tile, on
// the persistent direct-load stream of gemm_dma.h (one 256 x 256 workgroup
// per CU), reading W and H in place; the tile never leaves registers -- its
// epilogue reduces each token column to a (max, sum exp) pair over each
// wave's 128 vocabulary rows, written as a partial.  A merge pass combines a
// token's partials into lse and forms the target logit z_{t,y_t} =
// h_t . W_{y_t} directly (one dot product).  No floating-point atomics are used, so results
// are bitwise reproducible.

#include "logits_epilogue.h"
#include "rbp_internal.h"

namespace {

using namespace rbp::lp;
using rbp::gemm::kLdsBytes;
using rbp::gemm::Tile;
using rbp::gemm::tile_stream;
using rbp::gemm::kKMajor;
using rbp::gemm::map_tile;
using rbp::gemm::Operand;

// Forward: per 256 x 256 tile and wave, the partial (max, sum exp) of each
// token column over the wave's 128 vocabulary rows, written by the lower lane
// half as 128 contiguous bytes per column block (partials [Vp/128][ld_part],
// token-contiguous); no exchange between the waves.
RBP_LOGITS_KERNEL void logits_lse_partial_kernel(const uint16_t* __restrict__ W,
                                                 const uint16_t* __restrict__ H, int64_t T,
                                                 int32_t d, int32_t V, int64_t tiles_m,
                                                 int64_t tiles_n, float2* __restrict__ part,
                                                 int64_t ld_part) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
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
    if (lane < 32) {
      const int64_t half = (int64_t)(tile.m0 >> 7) + GL::wm();
#pragma unroll
      for (int ni = 0; ni < GL::NI; ++ni)
        part[half * ld_part + tile.n0 + GL::col(ni)] = make_float2(mx[ni], sum[ni]);
    }
  };
  tile_stream<GL, kKMajor, kKMajor, kDeepLogits>(A, B, (int32_t)(tiles_m * tiles_n), smem,
                                                tile_of, epi);
}

// (m, s) <- merge with the partial (Mi, Si), rescaling to the larger max.
__device__ __forceinline__ void merge_ms(float& m, float& s, float Mi, float Si) {
  if (Mi == -INFINITY) return;  // a half tile past the vocabulary
  if (Mi > m) {
    s = fmaf(s, exp2f((m - Mi) * kLog2e), Si);
    m = Mi;
  } else {
    s = fmaf(Si, exp2f((Mi - m) * kLog2e), s);
  }
}

// 64 tokens per block of 16 waves.  Wave q merges the partials q, q + 16, ...
// of the block's tokens (consecutive lanes read consecutive tokens), the 16
// results are combined in a fixed order, then each wave forms the target
// logits of 4 tokens with one dot product each.
constexpr int kMergeTokens = 64;
constexpr int kMergeWaves = 16;

__global__ void __launch_bounds__(64 * kMergeWaves) lse_merge_kernel(
    const float2* __restrict__ part, int64_t ld_part, int32_t n_half,
    const uint16_t* __restrict__ H, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ seq, int64_t T, int32_t d,
    int32_t V, float* __restrict__ logp, float* __restrict__ lse) {
  __shared__ float sm[kMergeWaves][kMergeTokens], ss[kMergeWaves][kMergeTokens];
  __shared__ float sl[kMergeTokens];
  const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * kMergeTokens;
  const int64_t t = t0 + c;
  float m = -INFINITY, s = 0.0f;
  if (t < T) {
    int32_t i = q;
    for (; i + kMergeWaves < n_half; i += 2 * kMergeWaves) {
      const float2 a = part[(int64_t)i * ld_part + t];
      const float2 b = part[(int64_t)(i + kMergeWaves) * ld_part + t];
      merge_ms(m, s, a.x, a.y);
      merge_ms(m, s, b.x, b.y);
    }
    if (i < n_half) {
      const float2 a = part[(int64_t)i * ld_part + t];
      merge_ms(m, s, a.x, a.y);
    }
  }
  sm[q][c] = m;
  ss[q][c] = s;
  __syncthreads();
  if (threadIdx.x < kMergeTokens) {
    float M = -INFINITY, S = 0.0f;
#pragma unroll
    for (int k = 0; k < kMergeWaves; ++k) merge_ms(M, S, sm[k][c], ss[k][c]);
    const bool valid = t < T && (seq == nullptr || seq[t] >= 0);
    const float l = M + logf(S);
    sl[c] = valid ? l : 0.0f;
    if (t < T) lse[t] = valid ? l : 0.0f;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 0; k < kMergeTokens / kMergeWaves; ++k) {
    const int cc = q * (kMergeTokens / kMergeWaves) + k;
    const int64_t tt = t0 + cc;
    if (tt >= T) break;
    if (seq != nullptr && seq[tt] < 0) {
      if (lane == 0) logp[tt] = 0.0f;
      continue;
    }
    const int32_t y = tokens[tt];
    const bool y_ok = y >= 0 && y < V;
    const float z = dot_bf16_wave(H + tt * d, W + (int64_t)(y_ok ? y : 0) * d, d, lane);
    if (lane == 0) logp[tt] = y_ok ? z - sl[cc] : NAN;
  }
}

}  // namespace

size_t rbp::logprob_fwd_ws(int64_t T, int32_t V) {
  const int64_t n_half = round256(V) / 128;
  return align_up(sizeof(float2) * (size_t)round256(T < 1 ? 1 : T) * (size_t)n_half, 256);
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
  const int64_t ld_part = tiles_n * 256;
  const int64_t grid = rbp::gemm::stream_grid(tiles_m * tiles_n, device_cus());
  hipLaunchKernelGGL(logits_lse_partial_kernel, dim3(grid), dim3(GL::kThreads), 0, s, W,
                     hidden, T, d, V, tiles_m, tiles_n, part, ld_part);
  hipLaunchKernelGGL(lse_merge_kernel, dim3(rbp::ceil_div(T, kMergeTokens)),
                     dim3(64 * kMergeWaves), 0, s, part, ld_part, (int32_t)(tiles_m * 2), hidden,
                     W, tokens, seq_of_token, T, d, V, logp, lse);
  RBP_CHECK_LAUNCH("policy_logprob_fwd");
  return RBP_OK;
}
