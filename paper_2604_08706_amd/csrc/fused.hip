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
// tile pass's exponentials, taken against a per-token reference R_t chosen
// before the pass, so that dz becomes one scalar per token times the stored
// values.  Per chunk of Tc tokens:
//   0. R_t = z_{t,y_t} - old_logp_t, with the target logit as one dot
//      product: the log-sum-exp the behaviour policy's probability implies,
//      equal to lse_t - log rho_t (rho_t the importance ratio, close to 1 for
//      a replayed token);
//   1. Z^T = W H^T tile by tile.  For each token column and 128-row half tile
//      i (one wave's rows), the epilogue stores q = exp(z - R_t) as bf16 into
//      Q^T [Vp][Tc] (the layout the backward products read) and writes the
//      partial (M_i, S_i, E_i) = (R_t, sum q, sum q z) -- or, for a half tile
//      whose sums leave [2^-60, 2^28] (R_t too far from its logits) or whose
//      reference is NaN, M_i = max z, S_i = sum exp(z - M_i), E_i = sum
//      exp(z - M_i) z and q = exp(z - R_t), or q = exp(z - M_i) where that
//      would exceed exp(20) (M_i > R_t + 20): M_i is always the reference of
//      the half tile's sums;
//   2. merge: lse and entropy from the partials, logp from the target logit;
//      a token is "referenced" when R_t lies in [M_t - 20, M_t + 40], M_t the
//      largest reference of its partials (its largest logit whenever a half
//      tile was stored against its own maximum); the others -- a ratio below
//      about e^-20 or above about e^40, or an invalid behaviour log-prob --
//      are listed and take M_t as their reference instead;
//   3. the loss pass writes dlogp (policy_loss_fwd_bwd);
//   4. the listed tokens' columns of Q^T are re-referenced to M_t in place;
//      then per token c_t = -dlogp_t exp(ref_t - lse_t), so that
//      dz_{t,v} = c_t q_{t,v} off the target, and the target entry becomes
//      q_{t,y} = dz_{t,y} / c_t = exp(lse_t - ref_t) (p_{t,y} - 1); and
//      H' = c (.) H, row t of the hidden states scaled by c_t, in bf16;
//   5. dW (+)= Q H' (sum over tokens of q_t (c_t h_t)^T) and
//      dh_t = c_t (Q^T W)_t, the products of the 4-call backward with the
//      per-token scale folded into an operand and into an epilogue.
// Unlike policy_logprob_fwd this keeps a T x V array (2 V bytes per token, in
// the workspace): exp(z - R_t), the backward's dz up to one factor per token.
// dz is rounded to bf16 once, as q, and c_t h_t once more.

#include "logits_epilogue.h"
#include "rbp_internal.h"

namespace {

using namespace rbp::lp;
using rbp::gemm::kLdsBytes;
using rbp::gemm::map_tile;
using rbp::gemm::Operand;
using rbp::gemm::Tile;
using rbp::gemm::tile_stream;
using rbp::gemm::kKMajor;
using rbp::gemm::kKPaired;

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

// One 32-row block (mi) of the wave's q tile.  B is loaded with paired rows,
// so lane l holds tokens 2 (l % 32) and 2 (l % 32) + 1 (tiles ni = 0, 1) of the
// same 16 vocabulary rows: per row, e = exp(z - M) of both tokens go into
// their columns' sums (S, and E += e z when kEnt), and e f (f = exp(M - ref))
// is packed into one bf16 pair and stored as 4 bytes.  Lanes 0..31 then write
// 128 contiguous bytes of one row of Q^T and lanes 32..63 those of the row 4
// below: whole cache lines, with no exchange between lanes.  Rows past the
// vocabulary hold 0.
template <bool kFull, bool kEnt>
__device__ __forceinline__ void q_rows(const f32x16 (&acc)[GL::MI][GL::NI], const float (&ls)[2],
                                       const float (&f)[2], int mi, int32_t lim,
                                       __amdgpu_buffer_rsrc_t rQ, uint32_t off, int64_t ldQ,
                                       float (&S)[2], float (&E)[2]) {
  static_assert(GL::NI == 2, "two column tiles per wave");
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float q[2];
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      const float z = acc[mi][ni][r];
      q[ni] = exp2_hw(fmaf(z, kLog2e, -ls[ni]));
      if constexpr (!kFull)
        q[ni] = __uint_as_float(select_below(GL::row_off(mi, r), lim, __float_as_uint(q[ni]), 0u));
      S[ni] += q[ni];
      if constexpr (kEnt) E[ni] = fmaf(q[ni], z, E[ni]);
    }
    __builtin_amdgcn_raw_buffer_store_b32(pack_bf16x2(q[0] * f[0], q[1] * f[1]), rQ, off,
                                          (int)(GL::row_off(mi, r) * ldQ * 2), kStreamStore);
  }
}

// A half tile stores against the token's reference R_t unless its largest
// logit exceeds R_t by more than kRefAbove (q would pass exp(20)); a token
// keeps R_t as its reference when R_t is within [M_t - kRefAbove,
// M_t + kRefBelow] of the largest reference M_t of its partials (the top
// entries' q then stay in [exp(-47), exp(20)] and c_t = -dlogp_t rho_t stays
// finite).  The same fp32 comparison is made wherever the decision is needed.
constexpr float kRefAbove = 20.0f;
constexpr float kRefBelow = 40.0f;

__device__ __forceinline__ bool stores_against_ref(float m_half, float ref) {
  return m_half - ref <= kRefAbove;  // false for a NaN reference
}

// Step 0: the target logit z_{t,y_t} (one wave per token, fp32 dot product)
// and the reference R_t = z_{t,y_t} - old_logp_t for the tokens [0, T256);
// masked and padding tokens get R = 0 and z = 0, an invalid target id z = NaN.
// Also clears the count of tokens listed by the merge.
__global__ void __launch_bounds__(256) target_ref_kernel(
    const uint16_t* __restrict__ Hc, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ seq,
    const float* __restrict__ old_logp, int64_t Tn, int64_t T256, int32_t d, int32_t V,
    float* __restrict__ zy, float* __restrict__ R, int32_t* __restrict__ n_listed) {
  if (blockIdx.x == 0 && threadIdx.x == 0) *n_listed = 0;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T256) return;
  const bool valid = t < Tn && (seq == nullptr || seq[t] >= 0);
  float z = 0.0f, r = 0.0f;
  if (valid) {
    const int32_t y = tokens[t];
    z = (y >= 0 && y < V) ? dot_bf16_wave(Hc + t * d, W + (int64_t)y * d, d, lane) : NAN;
    r = z - old_logp[t];
  }
  if (lane == 0) {
    zy[t] = z;
    R[t] = r;
  }
}

// Step 1: logit tiles -> partials (M, S, E) per (half tile, token) and
// q = exp(z - M) f into Q^T, f = exp(M - R_t) for a half tile stored against
// the reference, else 1.  One exponential per logit: a max pass, then the
// store pass, which also sums exp(z - M) and, when the entropy is wanted
// (kEnt), exp(z - M) z.
template <bool kEnt>
RBP_LOGITS_KERNEL void logits_store_kernel(const uint16_t* __restrict__ W,
                                           const uint16_t* __restrict__ Hc, int64_t Tn,
                                           int32_t d, int32_t V, const float* __restrict__ Rc,
                                           float* __restrict__ pM, float* __restrict__ pS,
                                           float* __restrict__ pE, int64_t ldp,
                                           uint16_t* __restrict__ Qt, int64_t ldQ,
                                           int64_t tiles_m, int64_t tiles_n) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const Operand A{W, d, V, d};
  const Operand B{Hc, d, Tn, d};
  const int lane = threadIdx.x & 63;
  auto tile_of = [&](int32_t vid) {
    int32_t tm, tn;
    map_tile(vid, (int32_t)tiles_m, (int32_t)tiles_n, kGroupLogits, tm, tn);
    return Tile{tm * 256, tn * 256, 0, d};
  };
  // the references of this lane's token columns, loaded one tile ahead
  // (issued after an epilogue, used at the next one)
  float Rr[GL::NI];
  auto load_ref = [&](int32_t vid) {
    const Tile tile = tile_of(vid);
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni) Rr[ni] = Rc[tile.n0 + GL::col_paired(ni)];
  };
  load_ref((int32_t)blockIdx.x);
  const int32_t n_vid = (int32_t)(tiles_m * tiles_n);
  auto epi = [&](int32_t vid, f32x16 (&acc)[GL::MI][GL::NI]) {
    const Tile tile = tile_of(vid);
    const int32_t vlim = V - tile.m0;
    const int32_t lim = vlim - GL::row(0, 0);
    const auto rQ = __builtin_amdgcn_make_buffer_rsrc(
        uniform_ptr(Qt + (int64_t)tile.m0 * ldQ + tile.n0), 0, (int)(256 * ldQ * 2), 0x00020000);
    // lane l: row GL::row(0, 0), tokens 2 (l % 32) and 2 (l % 32) + 1
    const uint32_t off = (uint32_t)(GL::row(0, 0) * ldQ + GL::col_paired(0)) * 2u;
    // the partial of each of the lane's columns: reference (the exponent
    // offset of S, E and the stored q), S = sum exp(z - ref), E = sum exp(z - ref) z
    float ref[GL::NI], s[GL::NI], e[GL::NI];
    // Direct store against the token's reference: q = exp(z - R_t), no max
    // pass and no rescaling.  Kept when every column of the wave's half tile
    // has a sum in [2^-60, 2^28] (q <= 2^28 ~ e^19.4, and the half tile's
    // largest logit within ~47 of R_t); otherwise (or a NaN reference) the
    // half tile is redone below against its own maximum, overwriting q.
    bool direct = false;
    if (vlim >= 256) {
      const float ls[GL::NI] = {Rr[0] * kLog2e, Rr[1] * kLog2e};
      const float one[GL::NI] = {1.0f, 1.0f};
      float S[GL::NI] = {0.0f, 0.0f}, E[GL::NI] = {0.0f, 0.0f};
#pragma unroll
      for (int mi = 0; mi < GL::MI; ++mi)
        q_rows<true, kEnt>(acc, ls, one, mi, lim, rQ, off, ldQ, S, E);
      bool ok = true;
#pragma unroll
      for (int ni = 0; ni < GL::NI; ++ni) {
        s[ni] = S[ni] + __shfl_xor(S[ni], 32, 64);
        e[ni] = kEnt ? E[ni] + __shfl_xor(E[ni], 32, 64) : 0.0f;
        ref[ni] = Rr[ni];
        ok = ok && s[ni] >= 0x1p-60f && s[ni] <= 0x1p28f;  // false for NaN
      }
      direct = __all(ok);
    }
    if (!direct) {
      float mx[GL::NI];
      if (vlim >= 256)
        column_max<true>(acc, 0, mx);
      else
        column_max<false>(acc, lim, mx);
      // a half tile past the vocabulary has M = -inf: offset 0 keeps its
      // (discarded) exponentials finite, and f = exp(-inf) = 0
      float ls[GL::NI], f[GL::NI], S[GL::NI] = {0.0f, 0.0f}, E[GL::NI] = {0.0f, 0.0f};
#pragma unroll
      for (int ni = 0; ni < GL::NI; ++ni) {
        ls[ni] = mx[ni] == -INFINITY ? 0.0f : mx[ni] * kLog2e;
        f[ni] = stores_against_ref(mx[ni], Rr[ni]) ? exp2_hw((mx[ni] - Rr[ni]) * kLog2e) : 1.0f;
      }
#pragma unroll
      for (int mi = 0; mi < GL::MI; ++mi) {
        if (vlim >= 256)
          q_rows<true, kEnt>(acc, ls, f, mi, lim, rQ, off, ldQ, S, E);
        else
          q_rows<false, kEnt>(acc, ls, f, mi, lim, rQ, off, ldQ, S, E);
      }
#pragma unroll
      for (int ni = 0; ni < GL::NI; ++ni) {
        s[ni] = S[ni] + __shfl_xor(S[ni], 32, 64);
        e[ni] = kEnt ? E[ni] + __shfl_xor(E[ni], 32, 64) : 0.0f;
        ref[ni] = mx[ni];
      }
    }
    // both lane halves hold rows of the same columns; the lower half writes
    // the partials, 128 contiguous bytes per array and column block
    const int64_t half = (int64_t)(tile.m0 >> 7) + GL::wm();
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni) {
      if (lane < 32) {
        const int64_t o = half * ldp + tile.n0 + GL::col_paired(ni);
        pM[o] = ref[ni];
        pS[o] = s[ni];
        if (kEnt) pE[o] = e[ni];
      }
    }
    if (vid + (int32_t)gridDim.x < n_vid) load_ref(vid + (int32_t)gridDim.x);
  };
  tile_stream<GL, kKMajor, kKPaired, kDeepLogits>(A, B, n_vid, smem, tile_of, epi);
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
// consecutive tokens), the 16 results are combined in a fixed order by the
// first wave, which writes lse, logp (from the step-0 target logit), the
// entropy and the token's reference, and lists the tokens that cannot keep
// R_t (order-free: the fix-up treats each listed token on its own).
constexpr int kMergeTokens = 64;
constexpr int kMergeWaves = 16;

__global__ void __launch_bounds__(64 * kMergeWaves) fused_merge_kernel(
    const float* __restrict__ pM, const float* __restrict__ pS, const float* __restrict__ pE,
    int64_t ldp, int32_t n_half, const float* __restrict__ zy, const float* __restrict__ R,
    const int32_t* __restrict__ seq, int64_t Tn, float* __restrict__ logp,
    float* __restrict__ lse, float* __restrict__ ent, float* __restrict__ ref,
    int32_t* __restrict__ listed, int32_t* __restrict__ n_listed) {
  __shared__ float sm[kMergeWaves][kMergeTokens], ss[kMergeWaves][kMergeTokens],
      se[kMergeWaves][kMergeTokens];
  const int c = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * kMergeTokens + c;
  float m = -INFINITY, s = 0.0f, e = 0.0f;
  if (t < Tn) {
    int32_t i = q;
    // two partials per iteration: their loads are issued together
    // pE is read only when the entropy is wanted (the tile pass wrote it)
    for (; i + kMergeWaves < n_half; i += 2 * kMergeWaves) {
      const int64_t o0 = (int64_t)i * ldp + t, o1 = o0 + (int64_t)kMergeWaves * ldp;
      const float M0 = pM[o0], S0 = pS[o0], E0 = ent ? pE[o0] : 0.0f;
      const float M1 = pM[o1], S1 = pS[o1], E1 = ent ? pE[o1] : 0.0f;
      merge_partial(m, s, e, M0, S0, E0);
      merge_partial(m, s, e, M1, S1, E1);
    }
    if (i < n_half) {
      const int64_t o = (int64_t)i * ldp + t;
      merge_partial(m, s, e, pM[o], pS[o], ent ? pE[o] : 0.0f);
    }
  }
  sm[q][c] = m;
  ss[q][c] = s;
  se[q][c] = e;
  __syncthreads();
  if (threadIdx.x >= kMergeTokens || t >= Tn) return;
  float M = -INFINITY, S = 0.0f, E = 0.0f;
#pragma unroll
  for (int k = 0; k < kMergeWaves; ++k) merge_partial(M, S, E, sm[k][c], ss[k][c], se[k][c]);
  const bool valid = seq == nullptr || seq[t] >= 0;
  const float l = M + logf(S);
  lse[t] = valid ? l : 0.0f;
  logp[t] = valid ? zy[t] - l : 0.0f;
  if (ent != nullptr) ent[t] = valid ? l - E / S : 0.0f;
  const float r = R[t];
  const bool keeps = (M - r <= kRefAbove) && (r - M <= kRefBelow);  // false for NaN
  ref[t] = keeps ? r : M;
  if (valid && !keeps) listed[atomicAdd(n_listed, 1)] = (int32_t)t;
}

// Step 4a: the listed tokens' columns re-referenced to M_t in place.  Block b
// owns the 128 vocabulary rows of half tile b (one row per thread) and walks
// the list; each q is multiplied by exp(R_t - M_t) where its half tile was
// stored against R_t, else by exp(M_b - M_t).  Rows whose stored value
// underflowed stay 0 (their p is below exp(-87) of the reference's).
__global__ void __launch_bounds__(128) fixup_kernel(uint16_t* __restrict__ Qt, int64_t ldQ,
                                                    const float* __restrict__ pM, int64_t ldp,
                                                    const float* __restrict__ R,
                                                    const float* __restrict__ ref,
                                                    const int32_t* __restrict__ listed,
                                                    const int32_t* __restrict__ n_listed,
                                                    int64_t Tn, int32_t V) {
  const int32_t half = (int32_t)blockIdx.x;
  const int32_t v = half * 128 + (int32_t)threadIdx.x;
  int64_t n = *n_listed;
  if (n > Tn) n = Tn;
  for (int64_t i = 0; i < n; ++i) {
    const int64_t t = listed[i];
    const float Mb = pM[(int64_t)half * ldp + t], r = R[t], M = ref[t];
    const float x = stores_against_ref(Mb, r) ? fminf((r - M) * kLog2e, 126.0f)
                                              : (Mb - M) * kLog2e;
    const float fct = exp2_hw(x);
    if (v < V) {
      uint16_t* p = Qt + (int64_t)v * ldQ + t;
      *p = __builtin_bit_cast(uint16_t, (__bf16)(bf16_to_f32(*p) * fct));
    }
  }
}

// Step 4b: one block per token t < T256.  c_t = -dlogp_t exp(ref_t - lse_t)
// (0 for masked and padding tokens); H'_t = c_t h_t in bf16; the target
// entry q_{t,y} = exp(lse_t - ref_t) expm1(logp_t), so that c_t q_{t,y} =
// dlogp_t (1 - p_{t,y}).
__global__ void __launch_bounds__(256) token_scale_kernel(
    const uint16_t* __restrict__ Hc, const int32_t* __restrict__ tokens,
    const int32_t* __restrict__ seq, const float* __restrict__ lse,
    const float* __restrict__ logp, const float* __restrict__ dlogp,
    const float* __restrict__ ref, int64_t Tn, int32_t d, int32_t V, uint16_t* __restrict__ Hp,
    float* __restrict__ cs, uint16_t* __restrict__ Qt, int64_t ldQ) {
  const int64_t t = blockIdx.x;
  const bool valid = t < Tn && (seq == nullptr || seq[t] >= 0);
  const float c = valid ? -dlogp[t] * exp2_hw((ref[t] - lse[t]) * kLog2e) : 0.0f;
  uint4* dst = reinterpret_cast<uint4*>(Hp + t * d);
  const uint4* src = reinterpret_cast<const uint4*>(Hc + t * d);
  for (int32_t k = threadIdx.x; k < d / 8; k += 256) {
    uint4 o = make_uint4(0u, 0u, 0u, 0u);
    if (t < Tn) {
      const uint4 h = src[k];
      const uint32_t w[4] = {h.x, h.y, h.z, h.w};
      uint32_t r[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        r[j] = pack_bf16x2(c * bf16_to_f32((uint16_t)(w[j] & 0xffff)),
                           c * bf16_to_f32((uint16_t)(w[j] >> 16)));
      o = make_uint4(r[0], r[1], r[2], r[3]);
    }
    dst[k] = o;
  }
  if (threadIdx.x == 0) {
    cs[t] = c;
    if (valid) {
      const int32_t y = tokens[t];
      if (y >= 0 && y < V)
        Qt[(int64_t)y * ldQ + t] = __builtin_bit_cast(
            uint16_t, (__bf16)(exp2_hw((lse[t] - ref[t]) * kLog2e) * expm1f(logp[t])));
    }
  }
}

// Workspace: Q^T [Vp][Tc] bf16, partials M, S, E [Vp / 128][Tc] fp32, the
// per-token target logit, reference R, chosen reference and scale [Tc] fp32,
// the list of re-referenced tokens [Tc] and its count, H' [Tc][d] bf16, the
// second dhidden K half [Tc][d] fp32, the loss pass's partial sums.
struct FusedWs {
  uint16_t* Qt;
  float *pM, *pS, *pE;
  float *zy, *R, *ref, *cs;
  int32_t *listed, *n_listed;
  uint16_t* Hp;
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
  w.zy = c.take<float>((size_t)Tc);
  w.R = c.take<float>((size_t)Tc);
  w.ref = c.take<float>((size_t)Tc);
  w.cs = c.take<float>((size_t)Tc);
  w.listed = c.take<int32_t>((size_t)Tc);
  w.n_listed = c.take<int32_t>(1);
  w.Hp = c.take<uint16_t>((size_t)Tc * (size_t)d);
  w.dh_half = c.take<float>((size_t)Tc * (size_t)d);
  w.loss_bytes = rbp::loss_ws(Tc);
  w.loss = c.take<uint8_t>(w.loss_bytes);
  w.bytes = rbp::align_up(c.used, 256);
  return w;
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
  const int64_t Vp = round256(V), tiles_v = Vp / 256;
  const int n_cu = device_cus();
  hipError_t e = hipSuccess;
#define RBP_FUSED_MARK(k)                                                                 \
  do {                                                                                    \
    e = mark(exec, (k), s);                                                               \
    if (e != hipSuccess) {                                                                \
      rbp::set_error("policy_fused_fwd_bwd: recording phase event %d: %s", (k),           \
                     hipGetErrorString(e));                                               \
      return RBP_EHIP;                                                                    \
    }                                                                                     \
  } while (0)
  for (int64_t t0 = 0; t0 < T; t0 += Tc) {
    const int64_t Tn = (T - t0) < Tc ? (T - t0) : Tc;
    const int64_t T256 = round256(Tn), tiles_t = T256 / 256;
    const uint16_t* Hc = hidden + t0 * d;
    const int32_t* sq = seq_of_token + t0;
    RBP_FUSED_MARK(RBP_PHASE_START);
    hipLaunchKernelGGL(target_ref_kernel, dim3(rbp::ceil_div(T256, 4)), dim3(256), 0, s, Hc, W,
                       tokens + t0, sq, old_logp + t0, Tn, T256, d, V, w.zy, w.R, w.n_listed);
    hipLaunchKernelGGL(entropy ? logits_store_kernel<true> : logits_store_kernel<false>,
                       dim3(rbp::gemm::stream_grid(tiles_v * tiles_t, n_cu)),
                       dim3(GL::kThreads), 0, s, W, Hc, Tn, d, V, w.R, w.pM, w.pS, w.pE, Tc,
                       w.Qt, Tc, tiles_v, tiles_t);
    RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    RBP_FUSED_MARK(RBP_PHASE_LOGITS);
    hipLaunchKernelGGL(fused_merge_kernel, dim3(rbp::ceil_div(Tn, kMergeTokens)),
                       dim3(64 * kMergeWaves), 0, s, w.pM, w.pS, w.pE, Tc, (int32_t)(Vp / 128),
                       w.zy, w.R, sq, Tn, logp + t0, lse + t0, entropy ? entropy + t0 : nullptr,
                       w.ref, w.listed, w.n_listed);
    RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    RBP_FUSED_MARK(RBP_PHASE_MERGE);
    const int st = policy_loss_fwd_bwd(logp + t0, old_logp + t0, sq, adv, seq_len, Tn, B,
                                       n_seq_total, eps_low, eps_high, loss_accum, dlogp + t0,
                                       stats, w.loss, w.loss_bytes, stream);
    if (st != RBP_OK) return st;
    RBP_FUSED_MARK(RBP_PHASE_LOSS);
    hipLaunchKernelGGL(fixup_kernel, dim3((unsigned)(Vp / 128)), dim3(128), 0, s, w.Qt, Tc, w.pM,
                       Tc, w.R, w.ref, w.listed, w.n_listed, Tn, V);
    hipLaunchKernelGGL(token_scale_kernel, dim3((unsigned)T256), dim3(256), 0, s, Hc,
                       tokens + t0, sq, lse + t0, logp + t0, dlogp + t0, w.ref, Tn, d, V, w.Hp,
                       w.cs, w.Qt, Tc);
    RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    RBP_FUSED_MARK(RBP_PHASE_SCALE);
    const int acc = (accumulate_dW || t0 > 0) ? 1 : 0;
    // the dhidden K half is free until dhidden runs
    rbp::launch_dweight(w.Hp, w.Qt, Tc, Tn, d, V, dW, acc, 0, tiles_v, s, w.dh_half,
                        Tc * (int64_t)d);
    RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    RBP_FUSED_MARK(RBP_PHASE_DW);
    rbp::launch_dhidden(W, w.Qt, Tc, Tn, d, V, dhidden + t0 * d, w.dh_half, s, w.cs);
    RBP_CHECK_LAUNCH("policy_fused_fwd_bwd");
    RBP_FUSED_MARK(RBP_PHASE_DHIDDEN);
  }
#undef RBP_FUSED_MARK
  return RBP_OK;
}
