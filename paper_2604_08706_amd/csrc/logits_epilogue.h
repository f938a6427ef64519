// Device helpers shared by the log-prob products (logprob_fwd.hip,
// logprob_bwd.hip, fused.hip):
// the 8-wave tile grid, exponentials, per-column (max, sum exp) reductions of
// a 256 x 256 logit tile, wave reductions, the target-logit dot product and the
// bf16 store of a tile into a vocabulary-major [v][t] array.
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

// The operand each product keeps in three LDS buffers (gemm_dma.h
// tile_stream; 1: A, 2: B), measured per product at the 7B head: the logit
// products W (A), dW the hidden states (A), dhidden dz^T (B).
constexpr int kDeepLogits = 1;
constexpr int kDeepDw = 1;
constexpr int kDeepDh = 2;

// 2^x on the hardware unit (v_exp_f32, ~1 ulp).  Arguments here are
// (z - max) * log2 e <= 0; below -126 the result flushes toward zero, which
// only drops terms under 2^-126 of the largest one in a sum.
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __uint_as_float((uint32_t)b << 16);
}

// Two floats rounded to bf16 (nearest even) and packed, lo in the low half:
// one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
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

// Cache policy of the dz^T stores: non-temporal (cache-policy bits 2).  32
// tiles per XCD write 4 MB per round -- the whole L2 -- and, cached normally,
// would evict the operand rows the next tiles share (measured: 1.1 ms of 15.5
// at T=16384, V=152064).
constexpr int kStreamStore = 2;

// One 32-row block (mi) of the wave's tile of dz = -dlogp p, stored into the
// vocabulary-major array Gt[v][t].  B is loaded with paired rows
// (gemm_dma.h, kKPaired), so lane l holds tokens 2 (l % 32) and
// 2 (l % 32) + 1 (tiles ni = 0, 1) of the same 16 vocabulary rows: per row the
// two values are packed into one bf16 pair and stored as 4 bytes, lanes 0..31
// writing 128 contiguous bytes of one row and lanes 32..63 those of the row
// 4 below -- whole cache lines, with no exchange between lanes.  Stores go
// through a per-tile buffer resource (32-bit offsets from the tile's corner).
// Rows past the vocabulary hold zeros.
template <bool kFull>
__device__ __forceinline__ void dz_rows(const f32x16 (&acc)[GL::MI][GL::NI], const float (&ls)[2],
                                        const float (&dl)[2], int mi, int32_t lim,
                                        __amdgpu_buffer_rsrc_t rGt, uint32_t off, int64_t ldGt) {
  static_assert(GL::NI == 2, "two column tiles per wave");
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float g[2];
#pragma unroll
    for (int ni = 0; ni < 2; ++ni) {
      g[ni] = -dl[ni] * exp2_hw(fmaf(acc[mi][ni][r], kLog2e, -ls[ni]));
      if constexpr (!kFull)
        g[ni] = __uint_as_float(select_below(GL::row_off(mi, r), lim, __float_as_uint(g[ni]), 0u));
    }
    __builtin_amdgcn_raw_buffer_store_b32(pack_bf16x2(g[0], g[1]), rGt, off,
                                          (int)(GL::row_off(mi, r) * ldGt * 2), kStreamStore);
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
