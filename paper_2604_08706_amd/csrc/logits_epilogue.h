// Device helpers shared by the log-prob products (logprob_fwd.hip,
// logprob_bwd.hip, fused.hip):
// the 8-wave tile grid, exponentials, per-column (max, sum exp) reductions of
// a 256 x 256 logit tile, wave reductions, the target-logit dot product and the
// transposing bf16 store of a tile into a vocabulary-major [v][t] array.
#pragma once

#include <cmath>

#include "gemm_core.h"
#include "gemm_dma.h"

namespace rbp {
namespace lp {

using rbp::gemm::f32x16;

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kGroupLogits = 4;
constexpr int kGroupGrad = 8;   // dhidden: groups of 8 hidden-unit tiles
// dW: groups of 14 hidden-unit tiles, all of them at d = 3584, so that an
// XCD's concurrent tiles read each vocabulary panel of dz^T together
constexpr int kGroupDw = 14;

// Every product runs on the 8-wave grid (two waves per SIMD).
using GL = rbp::gemm::Grid8;
#define RBP_LOGITS_KERNEL                                                        \
  __global__ __attribute__((amdgpu_flat_work_group_size(GL::kThreads, GL::kThreads), \
                            amdgpu_waves_per_eu(GL::kWaves / 4, GL::kWaves / 4)))

// 2^x on the hardware unit (v_exp_f32, ~1 ulp).  Arguments here are
// (z - max) * log2 e <= 0; below -126 the result flushes toward zero, which
// only drops terms under 2^-126 of the largest one in a sum.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const __bf16 a = (__bf16)lo, b = (__bf16)hi;
  return (uint32_t)__builtin_bit_cast(uint16_t, a) | ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// a where off < lim, else b, as (a & mask) | (b & ~mask) with mask = all ones
// where off - lim < 0: three vector instructions in assembly.  A plain
// compare would become a lane mask in scalar registers (64 of them live at
// once overflow the scalar file), and a plain subtraction would be computed
// once and kept live for every later use (64 values per pass over a tile);
// volatile, so that every use forms its own difference and mask.
__device__ __forceinline__ uint32_t select_below(int off, int32_t lim, uint32_t a, uint32_t b) {
  int32_t d;
  uint32_t m, r;
  asm volatile("v_sub_u32 %0, %1, %2" : "=v"(d) : "i"(off), "v"(lim));
  asm volatile("v_ashrrev_i32 %0, 31, %1" : "=v"(m) : "v"(d));
  asm volatile("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(m), "v"(a), "v"(b));
  return r;
}

// acc, or -inf where the row is past the vocabulary (row_off >= lim): mask
// arithmetic rather than compares, whose masks would pile up in scalar
// registers.
template <bool kFull>
__device__ __forceinline__ float logit_or_ninf(float v, int off, int32_t lim) {
  if constexpr (kFull) return v;
  return __uint_as_float(select_below(off, lim, __float_as_uint(v), 0xff800000u));
}

// Per token column of this wave's 128 x 64 block: max and sum exp(z - max)
// over the lane pair's rows (lanes l and l + 32 hold the same column).
template <bool kFull>
__device__ __forceinline__ void column_stats(const f32x16 (&acc)[GL::MI][GL::NI], int32_t lim,
                                             float (&mx)[GL::NI], float (&sum)[GL::NI]) {
#pragma unroll
  for (int ni = 0; ni < GL::NI; ++ni) {
    float m = -INFINITY;
#pragma unroll
    for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        m = fmaxf(m, logit_or_ninf<kFull>(acc[mi][ni][r], GL::row_off(mi, r), lim));
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    // a column with no real row (tail tile) has m = -inf: offset 0 keeps the
    // exponentials at exp(-inf) = 0 instead of NaN
    const float mb = (kFull || m != -INFINITY) ? m * kLog2e : 0.0f;
    float s4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int mi = 0; mi < GL::MI; ++mi)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        s4[r & 3] += exp2_hw(
            fmaf(logit_or_ninf<kFull>(acc[mi][ni][r], GL::row_off(mi, r), lim), kLog2e, -mb));
    float sm = (s4[0] + s4[1]) + (s4[2] + s4[3]);
    sm += __shfl_xor(sm, 32, 64);
    mx[ni] = m;
    sum[ni] = sm;
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

// h . w over d bf16 elements (d % 8 == 0), one wave cooperating; every lane
// returns the full sum.
__device__ __forceinline__ float dot_bf16_wave(const uint16_t* __restrict__ h,
                                               const uint16_t* __restrict__ w, int32_t d,
                                               int lane) {
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
  return wave_sum(z);
}

// A pointer every lane holds the same value of, in scalar registers: buffer
// resources built from it need no per-lane loop.
template <class T>
__device__ __forceinline__ T* uniform_ptr(T* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return reinterpret_cast<T*>(((uint64_t)hi << 32) | lo);
}

// Transposing tile store.  A lane holds four consecutive vocabulary rows
// v0..v0+3 of one token.  The four lanes of a quad (tokens t0..t0+3) transpose
// their 4 x 4 block with two lane exchanges (DPP quad permutes; 16-bit halves
// regrouped with byte permutes), after which lane j of the quad holds row
// v0 + j for tokens t0..t0+3: one 8-byte store (see dz_rows for the grouping
// into whole cache lines).  Stores go through a per-tile buffer resource, so
// every address is a 32-bit offset from the tile's corner.
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t quad_xor1(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xf, 0xf, false);  // [1,0,3,2]
}
__device__ __forceinline__ uint32_t quad_xor2(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xf, 0xf, false);  // [2,3,0,1]
}
// byte permute: selector byte k picks byte k of the result from
// {hi (bytes 4..7), lo (bytes 0..3)}
__device__ __forceinline__ uint32_t byte_perm(uint32_t hi, uint32_t lo, uint32_t sel) {
  return __builtin_amdgcn_perm(hi, lo, sel);
}

// Selectors of the quad transpose for lane position j = lane % 4.
struct QuadSel {
  uint32_t send1, pick, send2, w0, w1;
  __device__ __forceinline__ QuadSel() {
    const int j = threadIdx.x & 3;
    const bool lo2 = j < 2, ev = (j & 1) == 0;
    send1 = lo2 ? 0x07060504u : 0x03020100u;  // lanes 0, 1 send rows 2, 3
    pick = lo2 ? 0x03020100u : 0x07060504u;
    send2 = ev ? 0x07060302u : 0x05040100u;
    w0 = ev ? 0x05040100u : 0x03020504u;
    w1 = ev ? 0x07060100u : 0x03020706u;
  }
};

// Cache policy of the dz^T stores: non-temporal.  32 tiles per XCD write 4 MB
// per round -- the whole L2 -- and, cached normally, would evict the operand
// rows the next tiles share (measured: 1.1 ms of 15.5 at T=16384, V=152064).
#ifndef RBP_QSTORE_CPOL
#define RBP_QSTORE_CPOL 2
#endif
constexpr int kStreamStore = RBP_QSTORE_CPOL;

// -dl p -> bf16 for four consecutive rows of one token, packed in pairs.
template <bool kFull>
__device__ __forceinline__ void dz_pack(const f32x16& acc, float ls, float dl, int mi, int rg,
                                        int32_t lim, uint32_t& P0, uint32_t& P1) {
  float g[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    g[i] = -dl * exp2_hw(fmaf(acc[rg * 4 + i], kLog2e, -ls));
    if constexpr (!kFull)  // rows past the vocabulary hold zeros
      g[i] = __uint_as_float(select_below(GL::row_off(mi, rg * 4 + i), lim,
                                          __float_as_uint(g[i]), 0u));
  }
  P0 = pack_bf16x2(g[0], g[1]);
  P1 = pack_bf16x2(g[2], g[3]);
}

// 4 x 4 transpose inside each lane quad: in, lane j holds rows r..r+3 of
// token t0 + j as (P0 = rows r, r+1; P1 = rows r+2, r+3); out, row r + j of
// tokens t0..t0+3 as (w0 = tokens 0, 1; w1 = tokens 2, 3).
__device__ __forceinline__ void quad_transpose(uint32_t P0, uint32_t P1, const QuadSel& qs,
                                               uint32_t& w0, uint32_t& w1) {
  // step 1 (partner j ^ 2): lanes 0, 1 keep rows r, r+1 and get their
  // partner's; lanes 2, 3 keep rows r+2, r+3.  A / B = this row pair for
  // tokens (j & 1) and (j & 1) + 2.
  const uint32_t r1 = quad_xor2(byte_perm(P1, P0, qs.send1));
  const uint32_t Ah = byte_perm(r1, P0, qs.pick);
  const uint32_t Bh = byte_perm(P1, r1, qs.pick);
  // step 2 (partner j ^ 1): even lanes collect the first row of the pair,
  // odd lanes the second
  const uint32_t r2 = quad_xor1(byte_perm(Bh, Ah, qs.send2));
  w0 = byte_perm(r2, Ah, qs.w0);
  w1 = byte_perm(r2, Bh, qs.w1);
}

// One 32-row block of both 32-token column blocks of a wave (NI == 2).
// Lanes 0..31 hold rows 0..3 (+8 rg) of their token, lanes 32..63 rows 4..7;
// a lane-half swap (v_permlane32_swap) first regroups them so that lanes
// 0..31 hold the first column block and lanes 32..63 the second, for the
// same four rows: each store then writes 4 rows x 128 contiguous bytes, whole
// cache lines.
template <bool kFull>
__device__ __forceinline__ void dz_rows(const f32x16 (&acc)[GL::MI][GL::NI], const float (&ls)[2],
                                        const float (&dl)[2], int mi, int32_t lim,
                                        const QuadSel& qs, __amdgpu_buffer_rsrc_t rGt,
                                        uint32_t off, int64_t ldGt) {
  static_assert(GL::NI == 2, "two column blocks per wave");
#pragma unroll
  for (int rg = 0; rg < 4; ++rg) {
    uint32_t X0, X1, Y0, Y1;  // column block 0 / 1, rows (0,1) / (2,3) of the lane's half
    dz_pack<kFull>(acc[mi][0], ls[0], dl[0], mi, rg, lim, X0, X1);
    dz_pack<kFull>(acc[mi][1], ls[1], dl[1], mi, rg, lim, Y0, Y1);
    const auto s0 = __builtin_amdgcn_permlane32_swap(X0, Y0, false, false);
    const auto s1 = __builtin_amdgcn_permlane32_swap(X1, Y1, false, false);
    // s0[0], s1[0]: rows 0..3 of the group; s0[1], s1[1]: rows 4..7
    uint32_t w0, w1;
    const int ro = mi * 32 + rg * 8;  // first row of the 8-row group within the wave's block
    quad_transpose(s0[0], s1[0], qs, w0, w1);
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{w0, w1}, rGt, off, (int)(ro * ldGt * 2), kStreamStore);
    quad_transpose(s0[1], s1[1], qs, w0, w1);
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{w0, w1}, rGt, off, (int)((ro + 4) * ldGt * 2),
                                          kStreamStore);
  }
}

inline int64_t round256(int64_t x) { return (x + 255) / 256 * 256; }

// Compute units of the current device (the persistent products launch one
// workgroup per CU).
inline int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
    n = 256;
  return n;
}

}  // namespace lp
}  // namespace rbp
