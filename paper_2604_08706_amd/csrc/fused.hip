// Single-pass log-prob forward, GRPO loss and log-prob backward
// (policy_fused_fwd_bwd), plus the per-token policy entropy.
//
// Same mathematics as policy_logprob_fwd + policy_loss_fwd_bwd +
// policy_logprob_bwd (App. D.2): z_t = W h_t, lse_t, logp_t = z_{t,y_t} - lse_t,
// the clipped objective's dlogp_t, dz_t = dlogp_t (e_{y_t} - p_t), dh_t = W^T dz_t,
// dW (+)= sum_t dz_t h_t^T; and H_t = -sum_v p log p = lse_t - sum_v p_{t,v} z_{t,v},
// the training entropy the paper tracks (App. E).
//
// The 4-call path recomputes the logit product in its backward, 8 d V flop per
// token; this path executes the 6 d V of the definition by keeping the forward
// tile pass's exponentials.  Per chunk of Tc tokens:
//   1. Z^T = W H^T tile by tile.  For each token column and 128-row half tile
//      i (one wave's rows), the epilogue writes the partial M_i = max z,
//      S_i = sum exp(z - M_i), E_i = sum exp(z - M_i) z, and stores
//      q = exp(z - M_i) as bf16 into Q^T [Vp][Tc] -- the layout the backward
//      products read (dz^T);
//   2. merge: lse and entropy from the partials, logp from one target dot
//      product;
//   3. the loss pass writes dlogp (policy_loss_fwd_bwd);
//   4. in place, q -> dz = -dlogp_t exp(M_i - lse_t) q, and each token's target
//      entry -> dlogp_t (1 - exp(logp_t)) from the fp32 logp;
//   5. dhidden and dW, the products of the 4-call backward.
// Unlike policy_logprob_fwd this keeps a T x V array (2 V bytes per token, in
// the workspace).  dz is rounded to bf16 twice (q, then the scaled value)
// instead of once.

#include "logits_epilogue.h"
#include "rbp_internal.h"

namespace {

using namespace rbp::lp;
using rbp::gemm::kLdsBytes;
using rbp::gemm::map_tile;
using rbp::gemm::Operand;
using rbp::gemm::Tile;
using rbp::gemm::tile_stream;

// Per token column of this wave's 128 x 64 block: the max over the lane
// pair's rows (lanes l and l + 32 hold the same column).
template <bool kFull>
__device__ __forceinline__ void column_max(const f32x16 (&acc)[GL::MI][GL::NI], int32_t lim,
                                           float (&mx)[GL::NI]) {
#pragma unroll
  for (int ni = 0; ni < GL::NI; ++ni) {
    float m = -INFINITY;
#pragma unroll
    for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        m = fmaxf(m, logit_or_ninf<kFull>(acc[mi][ni][r], GL::row_off(mi, r), lim));
    mx[ni] = fmaxf(m, __shfl_xor(m, 32, 64));
  }
}

// q = exp(z - M) for four consecutive rows of one token, packed to bf16 pairs;
// the fp32 q and q z are added to the column's sums (rows past the vocabulary
// hold q = 0).
template <bool kFull>
__device__ __forceinline__ void q_pack(const f32x16& acc, float ls, int mi, int rg, int32_t lim,
                                       uint32_t& P0, uint32_t& P1, float& S, float& E) {
  float q[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float z = acc[rg * 4 + i];
    q[i] = exp2_hw(fmaf(z, kLog2e, -ls));
    if constexpr (!kFull)
      q[i] = __uint_as_float(select_below(GL::row_off(mi, rg * 4 + i), lim,
                                          __float_as_uint(q[i]), 0u));
    S += q[i];
    E = fmaf(q[i], z, E);
  }
  P0 = pack_bf16x2(q[0], q[1]);
  P1 = pack_bf16x2(q[2], q[3]);
}

// dz_rows of the backward with q in place of dz, plus the sums.
template <bool kFull>
__device__ __forceinline__ void q_rows(const f32x16 (&acc)[GL::MI][GL::NI], const float (&ls)[2],
                                       int mi, int32_t lim, const QuadSel& qs,
                                       __amdgpu_buffer_rsrc_t rQ, uint32_t off, int64_t ldQ,
                                       float (&S)[2], float (&E)[2]) {
  static_assert(GL::NI == 2, "two column blocks per wave");
#pragma unroll
  for (int rg = 0; rg < 4; ++rg) {
    uint32_t X0, X1, Y0, Y1;
    q_pack<kFull>(acc[mi][0], ls[0], mi, rg, lim, X0, X1, S[0], E[0]);
    q_pack<kFull>(acc[mi][1], ls[1], mi, rg, lim, Y0, Y1, S[1], E[1]);
    const auto s0 = __builtin_amdgcn_permlane32_swap(X0, Y0, false, false);
    const auto s1 = __builtin_amdgcn_permlane32_swap(X1, Y1, false, false);
    uint32_t w0, w1;
    const int ro = mi * 32 + rg * 8;
    quad_transpose(s0[0], s1[0], qs, w0, w1);
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{w0, w1}, rQ, off, (int)(ro * ldQ * 2), kStreamStore);
    quad_transpose(s0[1], s1[1], qs, w0, w1);
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{w0, w1}, rQ, off, (int)((ro + 4) * ldQ * 2),
                                          kStreamStore);
  }
}

// Step 1: logit tiles -> partials (M, S, E) per (half tile, token) and
// q = exp(z - M) into Q^T.  One exponential per logit: a max pass, then the
// store pass, which also sums q and q z.
RBP_LOGITS_KERNEL void logits_store_kernel(const uint16_t* __restrict__ W,
                                           const uint16_t* __restrict__ Hc, int64_t Tn,
                                           int32_t d, int32_t V, float* __restrict__ pM,
                                           float* __restrict__ pS, float* __restrict__ pE,
                                           int64_t ldp, uint16_t* __restrict__ Qt, int64_t ldQ,
                                           int64_t tiles_m, int64_t tiles_n) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const Operand A{W, d, V, d};
  const Operand B{Hc, d, Tn, d};
  const QuadSel qs;
  const int lane = threadIdx.x & 63;
  const int j = threadIdx.x & 3;
  auto tile_of = [&](int32_t vid) {
    int32_t tm, tn;
    map_tile(vid, (int32_t)tiles_m, (int32_t)tiles_n, kGroupLogits, tm, tn);
    return Tile{tm * 256, tn * 256, 0, d};
  };
  auto epi = [&](int32_t vid, f32x16 (&acc)[GL::MI][GL::NI]) {
    const Tile tile = tile_of(vid);
    const int32_t vlim = V - tile.m0;
    const int32_t lim = vlim - GL::row(0, 0);
    float mx[GL::NI];
    if (vlim >= 256)
      column_max<true>(acc, 0, mx);
    else
      column_max<false>(acc, lim, mx);
    // a half tile past the vocabulary has M = -inf: offset 0 keeps its
    // (discarded) exponentials finite
    float ls[GL::NI], S[GL::NI] = {0.0f, 0.0f}, E[GL::NI] = {0.0f, 0.0f};
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni) ls[ni] = mx[ni] == -INFINITY ? 0.0f : mx[ni] * kLog2e;
    const auto rQ = __builtin_amdgcn_make_buffer_rsrc(
        uniform_ptr(Qt + (int64_t)tile.m0 * ldQ + tile.n0), 0, (int)(256 * ldQ * 2), 0x00020000);
    const uint32_t off =
        (uint32_t)((GL::wm() * (256 / GL::WM) + j) * ldQ + GL::wn() * (256 / GL::WN) +
                   32 * (lane >> 5) + ((lane & 31) - j)) * 2u;
#pragma unroll
    for (int mi = 0; mi < GL::MI; ++mi) {
      if (vlim >= 256)
        q_rows<true>(acc, ls, mi, lim, qs, rQ, off, ldQ, S, E);
      else
        q_rows<false>(acc, ls, mi, lim, qs, rQ, off, ldQ, S, E);
    }
    // both lane halves hold rows of the same columns; the lower half writes
    // the sums, 128 contiguous bytes per array and column block
    const int64_t half = (int64_t)(tile.m0 >> 7) + GL::wm();
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni) {
      const float s = S[ni] + __shfl_xor(S[ni], 32, 64);
      const float e = E[ni] + __shfl_xor(E[ni], 32, 64);
      if (lane < 32) {
        const int64_t o = half * ldp + tile.n0 + GL::col(ni);
        pM[o] = mx[ni];
        pS[o] = s;
        pE[o] = e;
      }
    }
  };
  tile_stream<GL, false, false>(A, B, (int32_t)(tiles_m * tiles_n), smem, tile_of, epi);
}

// (m, s, e) <- merge with the partial (Mi, Si, Ei), rescaling to the larger max.
__device__ __forceinline__ void merge_partial(float& m, float& s, float& e, float Mi, float Si,
                                              float Ei) {
  if (Mi == -INFINITY) return;  // a half tile past the vocabulary
  if (Mi > m) {
    const float f = exp2f((m - Mi) * kLog2e);
    s = fmaf(s, f, Si);
    e = fmaf(e, f, Ei);
    m = Mi;
  } else {
    const float f = exp2f((Mi - m) * kLog2e);
    s = fmaf(Si, f, s);
    e = fmaf(Ei, f, e);
  }
}

// Step 2: 64 tokens per block of 16 waves.  Wave q merges the partials
// i = q, q + 16, ... of the block's tokens (coalesced: consecutive lanes read
// consecutive tokens), the 16 results are combined in a fixed order, then
// each wave forms the target logits of 4 tokens with one dot product each.
constexpr int kMergeTokens = 64;
constexpr int kMergeWaves = 16;

__global__ void __launch_bounds__(64 * kMergeWaves) fused_merge_kernel(
    const float* __restrict__ pM, const float* __restrict__ pS, const float* __restrict__ pE,
    int64_t ldp, int32_t n_half, const uint16_t* __restrict__ Hc,
    const uint16_t* __restrict__ W, const int32_t* __restrict__ tokens,
    const int32_t* __restrict__ seq, int64_t Tn, int32_t d, int32_t V, float* __restrict__ logp,
    float* __restrict__ lse, float* __restrict__ ent) {
  __shared__ float sm[kMergeWaves][kMergeTokens], ss[kMergeWaves][kMergeTokens],
      se[kMergeWaves][kMergeTokens];
  __shared__ float sl[kMergeTokens];
  const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int64_t t0 = (int64_t)blockIdx.x * kMergeTokens;
  const int64_t t = t0 + c;
  float m = -INFINITY, s = 0.0f, e = 0.0f;
  if (t < Tn) {
    int32_t i = q;
    // two partials per iteration: their loads are issued together
    for (; i + kMergeWaves < n_half; i += 2 * kMergeWaves) {
      const int64_t o0 = (int64_t)i * ldp + t, o1 = o0 + (int64_t)kMergeWaves * ldp;
      const float M0 = pM[o0], S0 = pS[o0], E0 = pE[o0];
      const float M1 = pM[o1], S1 = pS[o1], E1 = pE[o1];
      merge_partial(m, s, e, M0, S0, E0);
      merge_partial(m, s, e, M1, S1, E1);
    }
    if (i < n_half) {
      const int64_t o = (int64_t)i * ldp + t;
      merge_partial(m, s, e, pM[o], pS[o], pE[o]);
    }
  }
  sm[q][c] = m;
  ss[q][c] = s;
  se[q][c] = e;
  __syncthreads();
  if (threadIdx.x < kMergeTokens) {
    float M = -INFINITY, S = 0.0f, E = 0.0f;
#pragma unroll
    for (int k = 0; k < kMergeWaves; ++k) merge_partial(M, S, E, sm[k][c], ss[k][c], se[k][c]);
    const bool valid = t < Tn && (seq == nullptr || seq[t] >= 0);
    const float l = M + logf(S);
    sl[c] = valid ? l : 0.0f;
    if (t < Tn) {
      lse[t] = valid ? l : 0.0f;
      if (ent != nullptr) ent[t] = valid ? l - E / S : 0.0f;
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int k = 0; k < kMergeTokens / kMergeWaves; ++k) {
    const int cc = q * (kMergeTokens / kMergeWaves) + k;
    const int64_t tt = t0 + cc;
    if (tt >= Tn) break;
    if (seq != nullptr && seq[tt] < 0) {
      if (lane == 0) logp[tt] = 0.0f;
      continue;
    }
    const int32_t y = tokens[tt];
    const bool y_ok = y >= 0 && y < V;
    const float z = dot_bf16_wave(Hc + tt * d, W + (int64_t)(y_ok ? y : 0) * d, d, lane);
    if (lane == 0) logp[tt] = y_ok ? z - sl[cc] : NAN;
  }
}

// Step 4: one block per (128 vocabulary rows, 2048 tokens), eight tokens per
// thread.  q -> -dlogp_t exp(M_i - lse_t) q in place; invalid tokens and the
// padding columns Tn..T256 become zero; then the target entries.
constexpr int kScaleTokens = 2048;

template <int kRows>
__device__ __forceinline__ void scale_rows(uint16_t* __restrict__ q, int64_t ldQ, int rows,
                                           const float (&c)[8]) {
#pragma unroll 8
  for (int r = 0; r < (kRows > 0 ? kRows : rows); ++r) {
    uint4* p = reinterpret_cast<uint4*>(q + r * ldQ);
    const uint4 x = *p;
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
    uint32_t o[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      o[k] = pack_bf16x2(c[2 * k] * bf16_to_f32((uint16_t)(w[k] & 0xffff)),
                         c[2 * k + 1] * bf16_to_f32((uint16_t)(w[k] >> 16)));
    *p = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

__global__ void __launch_bounds__(256) grad_scale_kernel(
    uint16_t* __restrict__ Qt, int64_t ldQ, int64_t T256, const float* __restrict__ pM,
    int64_t ldp, const float* __restrict__ lse, const float* __restrict__ logp,
    const float* __restrict__ dlogp, const int32_t* __restrict__ tokens,
    const int32_t* __restrict__ seq, int64_t Tn, int32_t V, int32_t group0) {
  const int64_t tb = (int64_t)blockIdx.x * kScaleTokens + threadIdx.x * 8;
  const int32_t group = group0 + (int32_t)blockIdx.y;  // 128-row vocabulary group
  const int32_t v0 = group * 128;
  const int32_t rows = V - v0 < 128 ? V - v0 : 128;
  if (tb >= T256 || rows <= 0) return;
  const float* m = pM + (int64_t)group * ldp + tb;
  float c[8], gy[8];
  int32_t y[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int64_t t = tb + k;
    const bool valid = t < Tn && (seq == nullptr || seq[t] >= 0);
    c[k] = 0.0f;
    gy[k] = 0.0f;
    y[k] = -1;
    if (valid) {
      const float dl = dlogp[t];
      c[k] = -dl * exp2_hw((m[k] - lse[t]) * kLog2e);
      gy[k] = -dl * expm1f(logp[t]);
      y[k] = tokens[t];
    }
  }
  uint16_t* q = Qt + (int64_t)v0 * ldQ + tb;
  if (rows == 128)
    scale_rows<128>(q, ldQ, rows, c);
  else
    scale_rows<0>(q, ldQ, rows, c);
  // the target rows, written after this thread's own scaled stores to them
#pragma unroll
  for (int k = 0; k < 8; ++k)
    if (y[k] >= v0 && y[k] < v0 + rows)
      q[(int64_t)(y[k] - v0) * ldQ + k] = __builtin_bit_cast(uint16_t, (__bf16)gy[k]);
}

// Workspace: Q^T [Vp][Tc] bf16, partials M, S, E [Vp / 128][Tc] fp32, the
// second dhidden K half [Tc][d] fp32, the loss pass's partial sums.
struct FusedWs {
  uint16_t* Qt;
  float *pM, *pS, *pE;
  float* dh_half;
  void* loss;
  size_t loss_bytes;
  size_t bytes;
};

FusedWs carve_fused(void* base, int64_t Tc, int32_t d, int32_t V) {
  rbp::WsCarver c(base);
  const int64_t Vp = round256(V);
  FusedWs w;
  w.Qt = c.take<uint16_t>((size_t)Vp * (size_t)Tc);
  w.pM = c.take<float>((size_t)(Vp / 128) * (size_t)Tc);
  w.pS = c.take<float>((size_t)(Vp / 128) * (size_t)Tc);
  w.pE = c.take<float>((size_t)(Vp / 128) * (size_t)Tc);
  w.dh_half = c.take<float>((size_t)Tc * (size_t)d);
  w.loss_bytes = rbp::loss_ws(Tc);
  w.loss = c.take<uint8_t>(w.loss_bytes);
  w.bytes = rbp::align_up(c.used, 256);
  return w;
}

// Vocabulary tiles of the first dW part: the smallest multiple of the tiles
// that make whole rounds of the persistent grid (tiles_d * tv0 % n_cu == 0)
// that is at least a fifth of the vocabulary -- the rescale of the rest, run
// beside it, then still finishes within it -- and leaves some tiles over; 0
// when no such split exists.
int64_t head_tiles(int64_t tiles_d, int64_t tiles_v, int n_cu) {
  int64_t a = tiles_d, b = n_cu;
  while (b != 0) {
    const int64_t r = a % b;
    a = b;
    b = r;
  }
  const int64_t step = n_cu / a;
  for (int64_t t = step; t < tiles_v; t += step)
    if (5 * t >= tiles_v) return t;
  return 0;
}

}  // namespace

size_t rbp::fused_ws(int64_t Tc, int32_t d, int32_t V) {
  return carve_fused(nullptr, round256(Tc < 1 ? 1 : Tc), d < 1 ? 1 : d, V < 1 ? 1 : V).bytes;
}

namespace {

// Records phase event k of `ex` (if given) on s.
inline hipError_t mark(const rbp_exec* ex, int k, hipStream_t s) {
  if (ex == nullptr || ex->phase_event[k] == nullptr) return hipSuccess;
  return hipEventRecord(reinterpret_cast<hipEvent_t>(ex->phase_event[k]), s);
}

}  // namespace

extern "C" int policy_fused_fwd_bwd(const uint16_t* hidden, const uint16_t* W,
                                    const int32_t* tokens, const int32_t* seq_of_token,
                                    const float* old_logp, const float* adv,
                                    const int32_t* seq_len, int64_t T, int32_t d, int32_t V,
                                    int32_t B, int64_t n_seq_total, float eps_low,
                                    float eps_high, float* logp, float* lse, float* entropy,
                                    float* loss_accum, float* dlogp, float* stats,
                                    float* dhidden, float* dW, int accumulate_dW, void* ws,
                                    size_t ws_bytes, const rbp_exec* exec, void* stream) {
  rbp::clear_error();
  RBP_REQUIRE(T >= 0 && d >= 1 && V >= 1, RBP_EINVAL,
              "policy_fused_fwd_bwd: need T >= 0, d >= 1, V >= 1");
  RBP_REQUIRE(d % 8 == 0, RBP_EUNSUPPORTED, "policy_fused_fwd_bwd: d %% 8 != 0 (d = %d)", d);
  RBP_REQUIRE(B >= 1 && n_seq_total >= 1, RBP_EINVAL,
              "policy_fused_fwd_bwd: need B >= 1 and n_seq_total >= 1");
  RBP_REQUIRE(eps_low >= 0.0f && eps_high >= 0.0f, RBP_EINVAL,
              "policy_fused_fwd_bwd: negative clip range");
  RBP_REQUIRE(W && dW && adv && seq_len && loss_accum && stats, RBP_EINVAL,
              "policy_fused_fwd_bwd: null pointer");
  RBP_REQUIRE(T == 0 || (hidden && tokens && seq_of_token && old_logp && logp && lse && dlogp &&
                         dhidden),
              RBP_EINVAL, "policy_fused_fwd_bwd: null per-token pointer");
  const bool overlap = exec != nullptr && exec->side_stream != nullptr;
  RBP_REQUIRE(!overlap || (exec->fork_event && exec->join_event), RBP_EINVAL,
              "policy_fused_fwd_bwd: a side stream needs both fork_event and join_event");
  RBP_REQUIRE(!overlap || exec->side_stream != stream, RBP_EINVAL,
              "policy_fused_fwd_bwd: the side stream must differ from `stream`");
  hipStream_t s = rbp::as_stream(stream);
  if (T == 0) {
    rbp::launch_grad_products(nullptr, W, nullptr, 0, 0, d, V, nullptr, nullptr, dW,
                              accumulate_dW, s);
    RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    return RBP_OK;
  }
  // largest chunk (multiple of 256 tokens, at most 2^21 so that every per-tile
  // byte range of Q^T fits a 32-bit buffer offset) whose workspace fits
  int64_t Tc = 0;
  if (ws) {
    int64_t lo = 256, hi = round256(T) < (int64_t(1) << 21) ? round256(T) : (int64_t(1) << 21);
    if (rbp::fused_ws(lo, d, V) <= ws_bytes) {
      while (lo < hi) {
        const int64_t mid = (lo + hi + 256) / 512 * 256;
        if (rbp::fused_ws(mid, d, V) <= ws_bytes) lo = mid; else hi = mid - 256;
      }
      Tc = lo;
    }
  }
  RBP_REQUIRE(Tc >= 256, RBP_EWORKSPACE,
              "policy_fused_fwd_bwd: workspace of %zu bytes holds no 256-token chunk (needs %zu)",
              ws_bytes, rbp::fused_ws(256, d, V));
  const FusedWs w = carve_fused(ws, Tc, d, V);
  hipStream_t side = overlap ? rbp::as_stream(exec->side_stream) : nullptr;
  hipEvent_t fork = overlap ? reinterpret_cast<hipEvent_t>(exec->fork_event) : nullptr;
  hipEvent_t join = overlap ? reinterpret_cast<hipEvent_t>(exec->join_event) : nullptr;
  const int64_t Vp = round256(V), tiles_v = Vp / 256;
  const int n_cu = device_cus();
  hipError_t e = hipSuccess;
#define RBP_FUSED_HIP(call)                                                               \
  do {                                                                                    \
    e = (call);                                                                           \
    if (e != hipSuccess) {                                                                \
      rbp::set_error("policy_fused_fwd_bwd: %s: %s", #call, hipGetErrorString(e));        \
      return RBP_EHIP;                                                                    \
    }                                                                                     \
  } while (0)
  for (int64_t t0 = 0; t0 < T; t0 += Tc) {
    const int64_t Tn = (T - t0) < Tc ? (T - t0) : Tc;
    const int64_t T256 = round256(Tn), tiles_t = T256 / 256;
    const uint16_t* Hc = hidden + t0 * d;
    const int32_t* sq = seq_of_token + t0;
    RBP_FUSED_HIP(mark(exec, RBP_PHASE_START, s));
    hipLaunchKernelGGL(logits_store_kernel, dim3(rbp::gemm::stream_grid(tiles_v * tiles_t, n_cu)),
                       dim3(GL::kThreads), 0, s, W, Hc, Tn, d, V, w.pM, w.pS, w.pE, Tc, w.Qt, Tc,
                       tiles_v, tiles_t);
    RBP_FUSED_HIP(mark(exec, RBP_PHASE_LOGITS, s));
    hipLaunchKernelGGL(fused_merge_kernel, dim3(rbp::ceil_div(Tn, kMergeTokens)),
                       dim3(64 * kMergeWaves), 0, s,
                       w.pM, w.pS, w.pE, Tc, (int32_t)(Vp / 128), Hc, W, tokens + t0, sq, Tn, d, V,
                       logp + t0, lse + t0, entropy ? entropy + t0 : nullptr);
    RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    RBP_FUSED_HIP(mark(exec, RBP_PHASE_MERGE, s));
    const int st = policy_loss_fwd_bwd(logp + t0, old_logp + t0, sq, adv, seq_len, Tn, B,
                                       n_seq_total, eps_low, eps_high, loss_accum, dlogp + t0,
                                       stats, w.loss, w.loss_bytes, stream);
    if (st != RBP_OK) return st;
    RBP_FUSED_HIP(mark(exec, RBP_PHASE_LOSS, s));
    const int acc = (accumulate_dW || t0 > 0) ? 1 : 0;
    const unsigned gx = (unsigned)rbp::ceil_div(T256, kScaleTokens);
    const int64_t tv0 = overlap ? head_tiles(rbp::ceil_div(d, 256), tiles_v, n_cu) : 0;
    if (tv0 > 0) {
      // rescale rows [0, 256 tv0); then, on the side stream, the rest while
      // dW runs over the first tv0 vocabulary tiles; dW of the rest and
      // dhidden once both parts are done
      const int32_t g0 = (int32_t)(tv0 * 2);  // 128-row groups in the head
      hipLaunchKernelGGL(grad_scale_kernel, dim3(gx, (unsigned)g0), dim3(256), 0, s, w.Qt, Tc,
                         T256, w.pM, Tc, lse + t0, logp + t0, dlogp + t0, tokens + t0, sq, Tn, V,
                         0);
      RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
      RBP_FUSED_HIP(mark(exec, RBP_PHASE_SCALE, s));
      RBP_FUSED_HIP(hipEventRecord(fork, s));
      RBP_FUSED_HIP(hipStreamWaitEvent(side, fork, 0));
      hipLaunchKernelGGL(grad_scale_kernel, dim3(gx, (unsigned)(Vp / 128 - g0)), dim3(256), 0,
                         side, w.Qt, Tc, T256, w.pM, Tc, lse + t0, logp + t0, dlogp + t0,
                         tokens + t0, sq, Tn, V, g0);
      RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
      RBP_FUSED_HIP(hipEventRecord(join, side));
      rbp::launch_dweight(Hc, w.Qt, Tc, Tn, d, V, dW, acc, 0, tv0, s);
      RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
      RBP_FUSED_HIP(hipStreamWaitEvent(s, join, 0));
      rbp::launch_dweight(Hc, w.Qt, Tc, Tn, d, V, dW, acc, tv0, tiles_v, s);
      RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    } else {
      hipLaunchKernelGGL(grad_scale_kernel, dim3(gx, (unsigned)(Vp / 128)), dim3(256), 0, s,
                         w.Qt, Tc, T256, w.pM, Tc, lse + t0, logp + t0, dlogp + t0, tokens + t0,
                         sq, Tn, V, 0);
      RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
      RBP_FUSED_HIP(mark(exec, RBP_PHASE_SCALE, s));
      rbp::launch_dweight(Hc, w.Qt, Tc, Tn, d, V, dW, acc, 0, tiles_v, s);
      RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    }
    RBP_FUSED_HIP(mark(exec, RBP_PHASE_DW, s));
    rbp::launch_dhidden(W, w.Qt, Tc, Tn, d, V, dhidden + t0 * d, w.dh_half, s);
    RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    RBP_FUSED_HIP(mark(exec, RBP_PHASE_DHIDDEN, s));
  }
#undef RBP_FUSED_HIP
  return RBP_OK;
}
