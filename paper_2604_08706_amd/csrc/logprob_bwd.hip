// Backward of the policy log-probabilities (policy_logprob_bwd) and the two
// gradient products shared with the single-pass entry.
//
// Paper: App. D.2, chain rule of logp_t = z_{t,y_t} - lse_t with z_t = W h_t:
//   dz_t = dlogp_t (e_{y_t} - softmax(z_t)),  dh_t = W^T dz_t,  dW = sum_t dz_t h_t^T.
//
// Per chunk of Tc tokens:
//   1. the forward's logit product is recomputed; its epilogue writes
//      dz = -dlogp p as bf16 into dz^T [Vp][Tc] (Vp = V rounded up to 256,
//      padding zero), and a small pass overwrites each token's target entry
//      with dlogp (1 - p_{t,y_t}) from a direct dot product for z_{t,y_t};
//   2. dH[t][m] = sum_v W[v][m] dz^T[v][t]: W and dz^T read MN-major;
//   3. dW[v][m] (+)= sum_t H[t][m] dz^T[v][t]: H read MN-major, dz^T K-major.
// Every product runs on the persistent direct-load stream of gemm_dma.h (one
// 256 x 256 workgroup per CU), reading W and H in place.  No floating-point
// atomics are used, so results are bitwise reproducible.

#include "logits_epilogue.h"
#include "rbp_internal.h"

namespace {

using namespace rbp::lp;
using rbp::gemm::kLdsBytes;
using rbp::gemm::Tile;
using rbp::gemm::tile_stream;
using rbp::gemm::map_tile;
using rbp::gemm::Operand;
using rbp::gemm::kKMajor;
using rbp::gemm::kMNMajor;
using rbp::gemm::kKPaired;

// Backward step 1: recompute the tile and write dz = dlogp (onehot - p) as
// bf16, vocabulary-major (Gt[v][t], the layout both later products read).
// The tile pass writes -dlogp_t p_{t,v} everywhere; the one target entry of
// each token is then overwritten by target_dz_kernel.  Masked and padding
// tokens get dz = 0 (p is evaluated against lse = +inf).

RBP_LOGITS_KERNEL void grad_logits_kernel(const uint16_t* __restrict__ W,
                                          const uint16_t* __restrict__ Hc, int64_t Tn,
                                          int32_t d, int32_t V, const int32_t* __restrict__ seq,
                                          const float* __restrict__ lse,
                                          const float* __restrict__ dlogp,
                                          uint16_t* __restrict__ Gt, int64_t ldGt,
                                          int64_t tiles_m, int64_t tiles_n) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const Operand A{W, d, V, d};
  const Operand B{Hc, d, Tn, d};
  auto tile_of = [&](int32_t vid) {
    int32_t tm, tn;
    map_tile(vid, (int32_t)tiles_m, (int32_t)tiles_n, kGroupLogits, tm, tn);
    return Tile{tm * 256, tn * 256, 0, d};
  };
  // lse * log2 e and dlogp of this lane's token columns, loaded one tile
  // ahead (issued after an epilogue, consumed at the next one)
  float ls[GL::NI], dl[GL::NI];
  auto load_token_terms = [&](int32_t vid) {
    const Tile tile = tile_of(vid);
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni) {
      const int64_t t = tile.n0 + GL::col_paired(ni);
      const bool valid = t < Tn && (seq == nullptr || seq[t] >= 0);
      ls[ni] = valid ? lse[t] * kLog2e : INFINITY;
      dl[ni] = valid ? dlogp[t] : 0.0f;
    }
  };
  load_token_terms((int32_t)blockIdx.x);
  const int32_t n_vid = (int32_t)(tiles_m * tiles_n);
  auto epi = [&](int32_t vid, f32x16 (&acc)[GL::MI][GL::NI]) {
    const Tile tile = tile_of(vid);
    const int32_t vlim = V - tile.m0;
    const int32_t lim = vlim - GL::row(0, 0);  // as row_off(mi, r) < lim
    // the tile's 256 x 256 corner of Gt
    const auto rGt = __builtin_amdgcn_make_buffer_rsrc(Gt + (int64_t)tile.m0 * ldGt + tile.n0, 0,
                                                       (int)(256 * ldGt * 2), 0x00020000);
    // lane l: row GL::row(0, 0), tokens 2 (l % 32) and 2 (l % 32) + 1
    const uint32_t off = (uint32_t)(GL::row(0, 0) * ldGt + GL::col_paired(0)) * 2u;
#pragma unroll
    for (int mi = 0; mi < GL::MI; ++mi) {
      if (vlim >= 256)
        dz_rows<true>(acc, ls, dl, mi, lim, rGt, off, ldGt);
      else
        dz_rows<false>(acc, ls, dl, mi, lim, rGt, off, ldGt);
    }
    if (vid + (int32_t)gridDim.x < n_vid) load_token_terms(vid + (int32_t)gridDim.x);
  };
  tile_stream<GL, kKMajor, kKPaired, kDeepLogits>(A, B, n_vid, smem, tile_of, epi);
}

// Backward step 1b, after the tile pass: the target entry of each valid
// token, dz_{t,y_t} = dlogp_t (1 - exp(z_{t,y_t} - lse_t)), with the target
// logit as one fp32 dot product h_t . W_{y_t}.  One wave per token.
__global__ void __launch_bounds__(256) target_dz_kernel(
    const uint16_t* __restrict__ Hc, const uint16_t* __restrict__ W,
    const int32_t* __restrict__ tokens, const int32_t* __restrict__ seq,
    const float* __restrict__ lse, const float* __restrict__ dlogp, int64_t Tn, int32_t d,
    int32_t V, uint16_t* __restrict__ Gt, int64_t ldGt) {
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= Tn || (seq != nullptr && seq[t] < 0)) return;
  const int32_t y = tokens[t];
  if (y < 0 || y >= V) return;
  const float z = dot_bf16_wave(Hc + t * d, W + (int64_t)y * d, d, lane);
  if (lane == 0) {
    const float p = exp2_hw((z - lse[t]) * kLog2e);
    const __bf16 g = (__bf16)(dlogp[t] * (1.0f - p));
    Gt[(int64_t)y * ldGt + t] = __builtin_bit_cast(uint16_t, g);
  }
}

// Backward step 2: dH[t][m] = c_t sum_v W[v][m] dz[t][v], with A = W and
// B = dz^T both read MN-major (m / t contiguous, k = vocabulary); c_t = 1,
// or cs[t] for the single pass.  The launch covers n_vid tiles from virtual
// tile vid_base on, over the whole vocabulary, or (split_steps > 0) each in
// two K halves of split_steps steps: virtual block 2 i + h is half h of tile
// vid_base + i; half 0 writes dH, half 1 its part[i] block ([t][m], 256 x
// 256 fp32), added by part_add_dh_kernel -- or, with part_full, its rows of
// part laid out like dH ([Tn][d]), added by add_f32_kernel.
RBP_LOGITS_KERNEL void dhidden_kernel(const uint16_t* __restrict__ W,
                                      const uint16_t* __restrict__ Gt, int64_t ldGt, int64_t Tn,
                                      int32_t d, int32_t V, const float* __restrict__ cs,
                                      float* __restrict__ dH, int64_t tiles_m, int64_t tiles_n,
                                      int32_t vid_base, int32_t n_vid, int32_t split_steps,
                                      float* __restrict__ part, int part_full) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const int64_t T256 = (Tn + 255) / 256 * 256;
  const Operand A{W, d, d, V};          // (m = hidden unit, k = vocab): W[v][m]
  const Operand B{Gt, ldGt, T256, V};   // (n = token, k = vocab): Gt[v][t]
  auto tile_of = [&](int32_t vid) {
    int32_t tm, tn;
    const int32_t half = split_steps > 0 ? (vid & 1) : 0;
    const int32_t tv = vid_base + (split_steps > 0 ? vid >> 1 : vid);
    map_tile(tv, (int32_t)tiles_m, (int32_t)tiles_n, kGroupGrad, tm, tn);
    // both halves span split_steps steps (uniform step count); columns past
    // V read as zero
    const int32_t kb = half * split_steps * 64;
    return Tile{tm * 256, tn * 256, kb, split_steps > 0 ? kb + split_steps * 64 : V};
  };
  auto epi = [&](int32_t vid, f32x16 (&acc)[GL::MI][GL::NI]) {
    const Tile tile = tile_of(vid);
    const bool to_part = split_steps > 0 && (vid & 1);
    float* blk = part + (int64_t)(vid >> 1) * 65536;
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni) {
      const int64_t t = tile.n0 + GL::col(ni);
      if (t >= Tn) continue;
      const float c = cs != nullptr ? cs[t] : 1.0f;  // per-token scale of the single pass
#pragma unroll
      for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int64_t m = tile.m0 + GL::row(mi, rg * 4);
          const float4 val = make_float4(c * acc[mi][ni][rg * 4 + 0], c * acc[mi][ni][rg * 4 + 1],
                                         c * acc[mi][ni][rg * 4 + 2], c * acc[mi][ni][rg * 4 + 3]);
          if (to_part && !part_full)
            *reinterpret_cast<float4*>(blk + GL::col(ni) * 256 + GL::row(mi, rg * 4)) = val;
          else if (m < d)
            *reinterpret_cast<float4*>((to_part ? part : dH) + t * d + m) = val;
        }
    }
  };
  tile_stream<GL, kMNMajor, kMNMajor, kDeepDh>(A, B, n_vid, smem, tile_of, epi);
}

// The last round of a dhidden launch when it is more than half full: its r
// tiles (virtual tiles vid_base .. vid_base + r - 1) are cut into s pieces
// of `steps` K steps each and run by one round of P = gridDim.x workgroups,
// with s - 1 = ceil(r / (P - r)).  Workgroup c < r runs pieces 0 .. s - 2 of
// tile c back to back, its accumulators carried from piece to piece, and
// writes dH; workgroup r + e runs the last piece of tiles e, e + (P - r),
// e + 2 (P - r), ... below r and writes each into part[i] (256 x 256 fp32,
// [t][m]), which part_add_dh_kernel adds afterwards.  No workgroup runs more
// than s - 1 pieces, so the round takes (s - 1) / s of a whole-vocabulary
// tile instead of leaving P - r compute units idle for all of it.  Virtual
// block vid = c + j P (j < s - 1) is workgroup c's j-th piece; the s r
// pieces are exactly the blocks below s r.
RBP_LOGITS_KERNEL void dhidden_pieces_kernel(const uint16_t* __restrict__ W,
                                             const uint16_t* __restrict__ Gt, int64_t ldGt,
                                             int64_t Tn, int32_t d, int32_t V,
                                             const float* __restrict__ cs,
                                             float* __restrict__ dH, int64_t tiles_m,
                                             int64_t tiles_n, int32_t vid_base, int32_t r,
                                             int32_t s, int32_t steps,
                                             float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const int64_t T256 = (Tn + 255) / 256 * 256;
  const Operand A{W, d, d, V};          // (m = hidden unit, k = vocab): W[v][m]
  const Operand B{Gt, ldGt, T256, V};   // (n = token, k = vocab): Gt[v][t]
  const int32_t P = (int32_t)gridDim.x;
  // tile i (of the round) and piece j of virtual block vid
  auto piece = [&](int32_t vid, int32_t& i, int32_t& j) {
    const int32_t c = vid % P, jj = vid / P;
    if (c < r) {
      i = c;
      j = jj;
    } else {
      i = jj * (P - r) + (c - r);
      j = s - 1;
    }
  };
  auto tile_of = [&](int32_t vid) {
    int32_t i, j, tm, tn;
    piece(vid, i, j);
    map_tile(vid_base + i, (int32_t)tiles_m, (int32_t)tiles_n, kGroupGrad, tm, tn);
    // every piece spans `steps` steps; columns past V read as zero
    const int32_t kb = j * steps * 64;
    return Tile{tm * 256, tn * 256, kb, kb + steps * 64};
  };
  auto epi = [&](int32_t vid, f32x16 (&acc)[GL::MI][GL::NI]) -> bool {
    int32_t i, j;
    piece(vid, i, j);
    if (j < s - 2) return false;  // the tile's next piece follows on this workgroup
    // dhidden_kernel's stores: c_t-scaled, the last piece into its block
    const Tile tile = tile_of(vid);
    const bool to_part = j == s - 1;
    float* blk = part + (int64_t)i * 65536;
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni) {
      const int64_t t = tile.n0 + GL::col(ni);
      if (t >= Tn) continue;
      const float c = cs != nullptr ? cs[t] : 1.0f;
#pragma unroll
      for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int64_t m = tile.m0 + GL::row(mi, rg * 4);
          const float4 val = make_float4(c * acc[mi][ni][rg * 4 + 0], c * acc[mi][ni][rg * 4 + 1],
                                         c * acc[mi][ni][rg * 4 + 2], c * acc[mi][ni][rg * 4 + 3]);
          if (to_part)
            *reinterpret_cast<float4*>(blk + GL::col(ni) * 256 + GL::row(mi, rg * 4)) = val;
          else if (m < d)
            *reinterpret_cast<float4*>(dH + t * d + m) = val;
        }
    }
    return true;
  };
  tile_stream<GL, kMNMajor, kMNMajor, kDeepDh>(A, B, s * r, smem, tile_of, epi);
}

// dH += part[i] over the tiles vid_base + i of a split dhidden launch; one
// block per (tile, 16 tokens).
__global__ void __launch_bounds__(256) part_add_dh_kernel(float* __restrict__ dH,
                                                          const float* __restrict__ part,
                                                          int32_t vid_base, int64_t tiles_m,
                                                          int64_t tiles_n, int32_t d,
                                                          int64_t Tn) {
  const int32_t i = (int32_t)blockIdx.x;
  int32_t tm, tn;
  map_tile(vid_base + i, (int32_t)tiles_m, (int32_t)tiles_n, kGroupGrad, tm, tn);
  const int32_t tl = (int32_t)blockIdx.y * 16 + (threadIdx.x >> 4);
  const int64_t t = (int64_t)tn * 256 + tl;
  if (t >= Tn) return;
  const float* src = part + (int64_t)i * 65536 + (int64_t)tl * 256;
  for (int32_t ml = (threadIdx.x & 15) * 4; ml < 256; ml += 64) {
    const int32_t m = tm * 256 + ml;
    if (m >= d) break;  // d % 8 == 0: a float4 never straddles the edge
    float4* dst = reinterpret_cast<float4*>(dH + t * d + m);
    const float4 p = *reinterpret_cast<const float4*>(src + ml);
    float4 o = *dst;
    o.x += p.x;
    o.y += p.y;
    o.z += p.z;
    o.w += p.w;
    *dst = o;
  }
}

// Backward step 3: dW[v][m] (+)= sum_t H[t][m] dz[t][v], with A = H read
// MN-major (m contiguous, k = token) and B = dz^T K-major (rows v, k = token).
// The launch covers n_vid of the tiles of the vocabulary range [tn_off,
// tn_off + tiles_n), from virtual tile vid_base on.  With split_steps > 0
// each of them is done in two K halves of split_steps steps (virtual block
// 2 i + h = half h of tile vid_base + i): half 0 updates dW, half 1 writes
// its raw sums to part[i] (a 256 x 256 fp32 block, [v][m]), which
// part_add_kernel adds afterwards -- the last, partly filled round of a
// persistent launch done as one round of half-length tiles.  Columns of dz^T
// past Tn are finite (the single pass) or zero, and meet zero rows of H.
RBP_LOGITS_KERNEL void dweight_kernel(const uint16_t* __restrict__ Hc,
                                      const uint16_t* __restrict__ Gt, int64_t ldGt, int64_t Tn,
                                      int32_t d, int32_t V, float* __restrict__ dW, int accumulate,
                                      int64_t tiles_m, int64_t tiles_n, int64_t tn_off,
                                      int32_t vid_base, int32_t n_vid, int32_t split_steps,
                                      float* __restrict__ part) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[kLdsBytes];
  const int64_t T8 = (Tn + 7) / 8 * 8;
  const Operand A{Hc, d, d, Tn};        // (m = hidden unit, k = token): H[t][m]
  const Operand B{Gt, ldGt, V, T8};     // (n = vocab, k = token): Gt[v][t]
  auto tile_of = [&](int32_t vid) {
    int32_t tm, tn;
    const int32_t half = split_steps > 0 ? (vid & 1) : 0;
    const int32_t tv = vid_base + (split_steps > 0 ? vid >> 1 : vid);
    map_tile(tv, (int32_t)tiles_m, (int32_t)tiles_n, kGroupDw, tm, tn);
    const int32_t kb = half * split_steps * 64;
    return Tile{tm * 256, (tn + (int32_t)tn_off) * 256, kb,
                split_steps > 0 ? kb + split_steps * 64 : (int32_t)Tn};
  };
  auto epi = [&](int32_t vid, f32x16 (&acc)[GL::MI][GL::NI]) {
    const Tile tile = tile_of(vid);
    if (split_steps > 0 && (vid & 1)) {
      float* blk = part + (int64_t)(vid >> 1) * 65536;
#pragma unroll
      for (int ni = 0; ni < GL::NI; ++ni)
#pragma unroll
        for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
          for (int rg = 0; rg < 4; ++rg)
            *reinterpret_cast<float4*>(blk + GL::col(ni) * 256 + GL::row(mi, rg * 4)) =
                make_float4(acc[mi][ni][rg * 4 + 0], acc[mi][ni][rg * 4 + 1],
                            acc[mi][ni][rg * 4 + 2], acc[mi][ni][rg * 4 + 3]);
      return;
    }
    if (accumulate && tile.n0 + 256 <= V && tile.m0 + 256 <= d) {
      // interior tile: the previous values are loaded kDwBatch float4 at a
      // time before any of them is stored back, so the tile waits for memory
      // a few times rather than once per float4 (batches of 4 and 16 time
      // the same)
      constexpr int kDwBatch = 8;
#pragma unroll
      for (int ni = 0; ni < GL::NI; ++ni) {
        float* row = dW + (int64_t)(tile.n0 + GL::col(ni)) * d + tile.m0;
#pragma unroll
        for (int mh = 0; mh < GL::MI; mh += kDwBatch / 4) {
          float4 o[kDwBatch];
#pragma unroll
          for (int k = 0; k < kDwBatch; ++k)
            o[k] = *reinterpret_cast<const float4*>(row + GL::row(mh + k / 4, (k % 4) * 4));
#pragma unroll
          for (int k = 0; k < kDwBatch; ++k) {
            const int mi = mh + k / 4, rg = k % 4;
            *reinterpret_cast<float4*>(row + GL::row(mi, rg * 4)) =
                make_float4(acc[mi][ni][rg * 4 + 0] + o[k].x, acc[mi][ni][rg * 4 + 1] + o[k].y,
                            acc[mi][ni][rg * 4 + 2] + o[k].z, acc[mi][ni][rg * 4 + 3] + o[k].w);
          }
          // keeps the next batch's loads below these stores (the compiler
          // would otherwise hoist them all and hold 16 float4 at once)
          asm volatile("" ::: "memory");
        }
      }
      return;
    }
#pragma unroll
    for (int ni = 0; ni < GL::NI; ++ni) {
      const int64_t v = tile.n0 + GL::col(ni);
      if (v >= V) continue;
#pragma unroll
      for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int64_t m = tile.m0 + GL::row(mi, rg * 4);
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
  };
  tile_stream<GL, kMNMajor, kKMajor, kDeepDw>(A, B, n_vid, smem, tile_of, epi);
}

// dW += part[i] over the tiles vid_base + i (i < n_tiles) of a split
// dweight launch; one block per (tile, 16 vocabulary rows).
__global__ void __launch_bounds__(256) part_add_kernel(float* __restrict__ dW,
                                                       const float* __restrict__ part,
                                                       int32_t vid_base, int64_t tiles_m,
                                                       int64_t tiles_n, int64_t tn_off,
                                                       int32_t d, int32_t V) {
  const int32_t i = (int32_t)blockIdx.x;
  int32_t tm, tn;
  map_tile(vid_base + i, (int32_t)tiles_m, (int32_t)tiles_n, kGroupDw, tm, tn);
  const int32_t m0 = tm * 256, v0 = (tn + (int32_t)tn_off) * 256;
  const int32_t vl = (int32_t)blockIdx.y * 16 + (threadIdx.x >> 4);
  const int32_t v = v0 + vl;
  if (v >= V) return;
  const float* src = part + (int64_t)i * 65536 + (int64_t)vl * 256;
  for (int32_t ml = (threadIdx.x & 15) * 4; ml < 256; ml += 64) {
    const int32_t m = m0 + ml;
    if (m >= d) break;  // d % 8 == 0: a float4 never straddles the edge
    float4* dst = reinterpret_cast<float4*>(dW + (int64_t)v * d + m);
    const float4 p = *reinterpret_cast<const float4*>(src + ml);
    float4 o = *dst;
    o.x += p.x;
    o.y += p.y;
    o.z += p.z;
    o.w += p.w;
    *dst = o;
  }
}

// a[i] += b[i] (n % 4 == 0), fixed order per element.
__global__ void __launch_bounds__(256) add_f32_kernel(float* __restrict__ a,
                                                      const float* __restrict__ b, int64_t n4) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4;
       i += (int64_t)gridDim.x * 256) {
    float4 x = reinterpret_cast<float4*>(a)[i];
    const float4 y = reinterpret_cast<const float4*>(b)[i];
    x.x += y.x;
    x.y += y.y;
    x.z += y.z;
    x.w += y.w;
    reinterpret_cast<float4*>(a)[i] = x;
  }
}

__global__ void __launch_bounds__(256) fill_zero_kernel(float* __restrict__ p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = 0.0f;
}



// Backward workspace carving: dz^T [Vp][T256] bf16, then the second dhidden
// K half [T256][d] fp32.
struct BwdWs {
  uint16_t* Gt;
  float* dh_half;
  size_t bytes;
};
BwdWs carve_bwd(void* base, int64_t Tc, int32_t d, int32_t V) {
  rbp::WsCarver c(base);
  const int64_t T256 = round256(Tc < 1 ? 1 : Tc), Vp = round256(V);
  BwdWs w;
  w.Gt = c.take<uint16_t>((size_t)Vp * (size_t)T256);
  w.dh_half = c.take<float>((size_t)T256 * (size_t)d);
  w.bytes = rbp::align_up(c.used, 256);
  return w;
}
}  // namespace

size_t rbp::logprob_bwd_ws(int64_t Tc, int32_t d, int32_t V) {
  return carve_bwd(nullptr, Tc, d < 1 ? 1 : d, V).bytes;
}

void rbp::launch_dweight(const uint16_t* Hc, const uint16_t* Gt, int64_t ldGt, int64_t Tn,
                         int32_t d, int32_t V, float* dW, int accumulate, int64_t tn_begin,
                         int64_t tn_end, hipStream_t s, float* scratch, int64_t scratch_floats) {
  const int64_t tiles_d = rbp::ceil_div(d, 256), tiles_n = tn_end - tn_begin;
  if (tiles_n <= 0) return;
  const int64_t tiles = tiles_d * tiles_n;
  const int64_t grid = rbp::gemm::stream_grid(tiles, device_cus());
  // A last round filled to at most half: its tiles go to a second launch as
  // two K halves each (one round of half the length), when the K range has
  // at least 8 steps and the scratch holds one 256 x 256 block per tile.
  const int64_t rem = tiles % grid, nk = rbp::ceil_div(Tn, 64);
  const bool split = tiles > grid && rem > 0 && 2 * rem <= grid && nk >= 8 &&
                     scratch != nullptr && rem * 65536 <= scratch_floats;
  const int64_t n_main = split ? tiles - rem : tiles;
  hipLaunchKernelGGL(dweight_kernel, dim3(grid), dim3(GL::kThreads), 0, s, Hc, Gt, ldGt, Tn, d,
                     V, dW, accumulate, tiles_d, tiles_n, tn_begin, 0, (int32_t)n_main, 0,
                     (float*)nullptr);
  if (!split) return;
  const int32_t half_steps = (int32_t)((nk + 1) / 2);
  hipLaunchKernelGGL(dweight_kernel, dim3(rbp::gemm::stream_grid(2 * rem, device_cus())),
                     dim3(GL::kThreads), 0, s, Hc, Gt, ldGt, Tn, d, V, dW, accumulate, tiles_d,
                     tiles_n, tn_begin, (int32_t)n_main, (int32_t)(2 * rem), half_steps, scratch);
  hipLaunchKernelGGL(part_add_kernel, dim3((unsigned)rem, 16), dim3(256), 0, s, dW, scratch,
                     (int32_t)n_main, tiles_d, tiles_n, tn_begin, d, V);
}

void rbp::launch_dhidden(const uint16_t* W, const uint16_t* Gt, int64_t ldGt, int64_t Tn,
                         int32_t d, int32_t V, float* dhidden_c, float* dh_half, hipStream_t s,
                         const float* cs) {
  const int n_cu = device_cus();
  const int64_t tiles_d = rbp::ceil_div(d, 256), tiles_t = rbp::ceil_div(Tn, 256);
  const int64_t tiles = tiles_d * tiles_t;
  const int64_t G = rbp::gemm::stream_grid(int64_t(1) << 30, n_cu);  // one round
  const int64_t nk = rbp::ceil_div(V, 64);
  const int32_t half_steps = (int32_t)((nk + 1) / 2);
  // The whole vocabulary per tile; when the tiles fill at most half a round,
  // all of them in two K halves (the second halves into dh_half, laid out
  // like dhidden, then summed); otherwise a last round filled to at most
  // half goes to a second launch as two K halves per tile (dh_half holds one
  // 256 x 256 block per tile).
  if (nk >= 8 && 2 * tiles <= G) {
    hipLaunchKernelGGL(dhidden_kernel, dim3(rbp::gemm::stream_grid(2 * tiles, n_cu)),
                       dim3(GL::kThreads), 0, s, W, Gt, ldGt, Tn, d, V, cs, dhidden_c, tiles_d,
                       tiles_t, 0, (int32_t)(2 * tiles), half_steps, dh_half, 1);
    const int64_t n4 = Tn * d / 4;
    int64_t blocks = rbp::ceil_div(n4, 256);
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(add_f32_kernel, dim3(blocks), dim3(256), 0, s, dhidden_c, dh_half, n4);
    return;
  }
  const int64_t r = tiles % G;
  const bool fits = r * 65536 <= ldGt * (int64_t)d;  // one scratch block per tile of the round
  const int64_t rem = (nk >= 8 && tiles > G && r > 0 && 2 * r <= G && fits) ? r : 0;
  // A last round more than half full: its tiles cut into pieces of the K
  // range, s - 1 = ceil(r / (G - r)) pieces per workgroup
  // (dhidden_pieces_kernel), when a piece keeps at least 8 steps and the
  // last piece is not empty.
  int64_t pieces = 0, piece_steps = 0;
  if (2 * r > G && fits) {
    const int64_t ps = 1 + rbp::ceil_div(r, G - r), st = rbp::ceil_div(nk, ps);
    if (ps <= 16 && st >= 8 && (ps - 1) * st < nk) {
      pieces = ps;
      piece_steps = st;
    }
  }
  const int64_t n_main = tiles - (rem > 0 ? rem : (pieces > 0 ? r : 0));
  if (n_main > 0)
    hipLaunchKernelGGL(dhidden_kernel, dim3(rbp::gemm::stream_grid(n_main, n_cu)),
                       dim3(GL::kThreads), 0, s, W, Gt, ldGt, Tn, d, V, cs, dhidden_c, tiles_d,
                       tiles_t, 0, (int32_t)n_main, 0, (float*)nullptr, 0);
  if (rem > 0) {
    hipLaunchKernelGGL(dhidden_kernel, dim3(rbp::gemm::stream_grid(2 * rem, n_cu)),
                       dim3(GL::kThreads), 0, s, W, Gt, ldGt, Tn, d, V, cs, dhidden_c, tiles_d,
                       tiles_t, (int32_t)n_main, (int32_t)(2 * rem), half_steps, dh_half, 0);
    hipLaunchKernelGGL(part_add_dh_kernel, dim3((unsigned)rem, 16), dim3(256), 0, s, dhidden_c,
                       dh_half, (int32_t)n_main, tiles_d, tiles_t, d, Tn);
  } else if (pieces > 0) {
    // grid G exactly: workgroup c's pieces are the virtual blocks c + j G
    hipLaunchKernelGGL(dhidden_pieces_kernel, dim3((unsigned)G), dim3(GL::kThreads), 0, s, W,
                       Gt, ldGt, Tn, d, V, cs, dhidden_c, tiles_d, tiles_t, (int32_t)n_main,
                       (int32_t)r, (int32_t)pieces, (int32_t)piece_steps, dh_half);
    hipLaunchKernelGGL(part_add_dh_kernel, dim3((unsigned)r, 16), dim3(256), 0, s, dhidden_c,
                       dh_half, (int32_t)n_main, tiles_d, tiles_t, d, Tn);
  }
}

void rbp::launch_grad_products(const uint16_t* Hc, const uint16_t* W, const uint16_t* Gt,
                               int64_t ldGt, int64_t Tn, int32_t d, int32_t V, float* dhidden_c,
                               float* dh_half, float* dW, int accumulate, hipStream_t s) {
  if (Tn == 0) {
    if (!accumulate) {
      const int64_t n = (int64_t)V * d;
      int64_t blocks = rbp::ceil_div(n, 256);
      if (blocks > 65536) blocks = 65536;
      hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, s, dW, n);
    }
    return;
  }
  launch_dhidden(W, Gt, ldGt, Tn, d, V, dhidden_c, dh_half, s);
  // dh_half is free again once dhidden's sum has read it
  launch_dweight(Hc, Gt, ldGt, Tn, d, V, dW, accumulate, 0, round256(V) / 256, s, dh_half,
                 ldGt * (int64_t)d);
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
  if (T == 0) {
    rbp::launch_grad_products(nullptr, W, nullptr, 0, 0, d, V, nullptr, nullptr, dW,
                              accumulate_dW, s);
    RBP_CHECK_LAUNCH("policy_logprob_bwd");
    return RBP_OK;
  }
  // largest chunk (multiple of 256 tokens) whose workspace fits
  int64_t Tc = 0;
  if (ws) {
    // chunks of at most 2^21 tokens keep every per-tile byte range of dz^T
    // (256 rows x Tc x 2 bytes) inside a 32-bit buffer offset
    int64_t lo = 256, hi = round256(T) < (int64_t(1) << 21) ? round256(T) : (int64_t(1) << 21);
    if (rbp::logprob_bwd_ws(lo, d, V) <= ws_bytes) {
      while (lo < hi) {  // largest multiple of 256 in [lo, hi] that fits
        const int64_t mid = (lo + hi + 256) / 512 * 256;
        if (rbp::logprob_bwd_ws(mid, d, V) <= ws_bytes) lo = mid; else hi = mid - 256;
      }
      Tc = lo;
    }
  }
  RBP_REQUIRE(Tc >= 256, RBP_EWORKSPACE,
              "policy_logprob_bwd: workspace of %zu bytes holds no 256-token chunk (needs %zu)",
              ws_bytes, rbp::logprob_bwd_ws(256, d, V));
  const BwdWs w = carve_bwd(ws, Tc, d, V);
  const int64_t tiles_v = round256(V) / 256;
  const int n_cu = device_cus();
  for (int64_t t0 = 0; t0 < T; t0 += Tc) {
    const int64_t Tn = (T - t0) < Tc ? (T - t0) : Tc;
    const int64_t tiles_t = rbp::ceil_div(Tn, 256);
    const uint16_t* Hc = hidden + t0 * d;
    hipLaunchKernelGGL(grad_logits_kernel, dim3(rbp::gemm::stream_grid(tiles_v * tiles_t, n_cu)),
                       dim3(GL::kThreads), 0, s, W, Hc, Tn, d, V,
                       seq_of_token ? seq_of_token + t0 : nullptr, lse + t0, dlogp + t0, w.Gt,
                       Tc, tiles_v, tiles_t);
    hipLaunchKernelGGL(target_dz_kernel, dim3(rbp::ceil_div(Tn, 4)), dim3(256), 0, s, Hc, W,
                       tokens + t0, seq_of_token ? seq_of_token + t0 : nullptr, lse + t0,
                       dlogp + t0, Tn, d, V, w.Gt, Tc);
    rbp::launch_grad_products(Hc, W, w.Gt, Tc, Tn, d, V, dhidden + t0 * d, w.dh_half, dW,
                              (accumulate_dW || t0 > 0) ? 1 : 0, s);
  }
  RBP_CHECK_LAUNCH("policy_logprob_bwd");
  return RBP_OK;
}
