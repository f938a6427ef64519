// bf16 MFMA tile machinery for gfx950 (CDNA4), shared by the three products of
// the log-prob path:  C[m][n] = sum_k A(m, k) * B(n, k), fp32 accumulation.
//
// Workgroup tile 256 x 256, K step 64, 256 threads = 4 waves in a 2 x 2 grid;
// each wave owns a 128 x 128 block = 4 x 4 v_mfma_f32_32x32x16_bf16 tiles
// (16 fp32 accumulators per lane each, 256 in total).
//
// Operands are staged HBM -> registers -> LDS, double buffered: the global
// loads of step k+1 are in flight while step k multiplies out of LDS.  An LDS
// operand tile is [256 rows (m or n)][64 k] bf16 = 8 chunks of 16 bytes per row
// with the chunk index XOR-swizzled by the row, so that
//   * a fragment read (32 consecutive rows, one chunk) and
//   * a transposing store (rows 8 apart, one chunk)
// both spread over all LDS banks.
//
// An operand stored "K-major" (k contiguous) is copied as is.  One stored
// "MN-major" (m or n contiguous) is read as 8 x 8 bf16 blocks and transposed in
// registers with byte permutes before the LDS store, so every product runs on
// the same fragment layout.
//
// MFMA 32x32x16 lane layout: lane l supplies A[l % 32][8 (l / 32) .. + 8) and
// B[l % 32][8 (l / 32) .. + 8) (k contiguous); accumulator r of lane l holds
// C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].  Hence each lane owns runs of four
// consecutive m for one n, which the epilogues store as 8/16-byte vectors.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace rbp {
namespace gemm {

typedef __bf16 bf16x8 __attribute__((__vector_size__(16)));
typedef float f32x16 __attribute__((__vector_size__(64)));
typedef uint32_t u32x4 __attribute__((__vector_size__(16)));

constexpr int kBM = 256, kBN = 256, kBK = 64;
constexpr int kThreads = 256;
constexpr int kTileBytes = 256 * kBK * 2;   // one operand tile, 32 KiB
constexpr int kStageBytes = 2 * kTileBytes; // A + B
constexpr int kLdsBytes = 2 * kStageBytes;  // double buffered, 128 KiB

// Stored operand: element (mn, k) is ptr[mn * ld + k] (K-major) or
// ptr[k * ld + mn] (MN-major).  Reads outside [0, mn_extent) x [0, k_extent)
// are replaced by zeros.  K-major operands need k_extent % 8 == 0, MN-major
// ones mn_extent % 8 == 0 (16-byte vectors never straddle the edge).
struct Operand {
  const uint16_t* ptr;
  int64_t ld;
  int64_t mn_extent;
  int64_t k_extent;
};

__device__ __forceinline__ int lds_off(int row, int chunk) {
  const int swz = (row ^ (row >> 3)) & 7;
  return row * 128 + ((chunk ^ swz) << 4);
}

// Global -> registers for one 256 x 64 operand tile.
template <bool KMAJOR>
__device__ __forceinline__ void load_tile(const Operand& op, int64_t mn0, int64_t k0,
                                          u32x4 (&r)[8]) {
  const int tid = threadIdx.x;
  if constexpr (KMAJOR) {
    // thread -> (row tid/8 + 32 p, chunk tid % 8): 8 lanes read one 128-byte row run
    const int64_t k = k0 + (tid & 7) * 8;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      const int64_t mn = mn0 + (tid >> 3) + 32 * p;
      if (mn < op.mn_extent && k < op.k_extent)
        r[p] = *reinterpret_cast<const u32x4*>(op.ptr + mn * op.ld + k);
      else
        r[p] = u32x4{0u, 0u, 0u, 0u};
    }
  } else {
    // thread -> 8 x 8 block (k rows kb*8.., mn columns mb*8..); 32 lanes read
    // 512 contiguous bytes of one k row
    const int kb = tid >> 5, mb = tid & 31;
    const int64_t mn = mn0 + mb * 8;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const int64_t k = k0 + kb * 8 + q;
      if (mn < op.mn_extent && k < op.k_extent)
        r[q] = *reinterpret_cast<const u32x4*>(op.ptr + k * op.ld + mn);
      else
        r[q] = u32x4{0u, 0u, 0u, 0u};
    }
  }
}

// Registers -> LDS tile (transposing MN-major blocks).
template <bool KMAJOR>
__device__ __forceinline__ void store_tile(const u32x4 (&r)[8], uint8_t* tile) {
  const int tid = threadIdx.x;
  if constexpr (KMAJOR) {
    const int chunk = tid & 7;
#pragma unroll
    for (int p = 0; p < 8; ++p)
      *reinterpret_cast<u32x4*>(tile + lds_off((tid >> 3) + 32 * p, chunk)) = r[p];
  } else {
    const int kb = tid >> 5, mb = tid & 31;
    // r[q] holds k row q, bf16 columns c = 0..7 (column c in dword c/2, half c%2).
    // Output row c gets, in dword q, (k = 2q, k = 2q + 1) of column c.
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
      u32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        o[q] = __builtin_amdgcn_perm(r[2 * q + 1][c >> 1], r[2 * q][c >> 1], sel);
      *reinterpret_cast<u32x4*>(tile + lds_off(mb * 8 + c, kb)) = o;
    }
  }
}

// One K step (64) of MFMAs for this wave out of one LDS stage.
__device__ __forceinline__ void mma_stage(const uint8_t* tA, const uint8_t* tB,
                                          f32x16 (&acc)[4][4]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int row = lane & 31;
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) {
    const int chunk = ks * 2 + (lane >> 5);
    bf16x8 a[4], b[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      a[i] = *reinterpret_cast<const bf16x8*>(tA + lds_off(wm * 128 + i * 32 + row, chunk));
      b[i] = *reinterpret_cast<const bf16x8*>(tB + lds_off(wn * 128 + i * 32 + row, chunk));
    }
#pragma unroll
    for (int mi = 0; mi < 4; ++mi)
#pragma unroll
      for (int ni = 0; ni < 4; ++ni)
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
  }
}

// Full K loop over [k_begin, k_end) for the tile at (m0, n0).  Ends with a
// barrier, so the caller may reuse `smem` right away.
template <bool A_KMAJOR, bool B_KMAJOR>
__device__ __forceinline__ void mainloop(const Operand& A, const Operand& B, int64_t m0,
                                         int64_t n0, int64_t k_begin, int64_t k_end,
                                         uint8_t* smem, f32x16 (&acc)[4][4]) {
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;
  const int64_t nk = (k_end - k_begin + kBK - 1) / kBK;
  if (nk <= 0) return;
  u32x4 ra[8], rb[8];
  load_tile<A_KMAJOR>(A, m0, k_begin, ra);
  load_tile<B_KMAJOR>(B, n0, k_begin, rb);
  store_tile<A_KMAJOR>(ra, smem);
  store_tile<B_KMAJOR>(rb, smem + kTileBytes);
  __syncthreads();
  for (int64_t it = 0; it < nk; ++it) {
    uint8_t* cur = smem + (it & 1) * kStageBytes;
    uint8_t* nxt = smem + ((it + 1) & 1) * kStageBytes;
    const bool more = it + 1 < nk;
    if (more) {
      const int64_t k = k_begin + (it + 1) * kBK;
      load_tile<A_KMAJOR>(A, m0, k, ra);
      load_tile<B_KMAJOR>(B, n0, k, rb);
    }
    mma_stage(cur, cur + kTileBytes, acc);
    if (more) {
      store_tile<A_KMAJOR>(ra, nxt);
      store_tile<B_KMAJOR>(rb, nxt + kTileBytes);
    }
    __syncthreads();
  }
}

// Block id -> (tile_m, tile_n).  The dispatcher hands block b to XCD b % 8, so
// blocks are first renumbered XCD by XCD (each XCD gets a contiguous range of
// tiles), then rastered in groups of `group_m` M-tiles per N-tile: the ~32
// blocks an XCD runs at once form a compact group_m x (32 / group_m) patch
// whose operand rows are shared through that XCD's L2.
__device__ __forceinline__ void map_tile(int64_t bid, int64_t tiles_m, int64_t tiles_n,
                                         int64_t group_m, int64_t& tm, int64_t& tn) {
  const int64_t nblk = tiles_m * tiles_n;
  const int64_t xcd = bid & 7, local = bid >> 3;
  const int64_t per = nblk >> 3, rem = nblk & 7;
  const int64_t L = xcd < rem ? xcd * (per + 1) + local
                              : rem * (per + 1) + (xcd - rem) * per + local;
  const int64_t group_size = group_m * tiles_n;
  const int64_t g = L / group_size;
  const int64_t first_m = g * group_m;
  const int64_t gm = (tiles_m - first_m) < group_m ? (tiles_m - first_m) : group_m;
  const int64_t in = L - g * group_size;
  tm = first_m + in % gm;
  tn = in / gm;
}

// Row (m) and column (n) of accumulator r of tile (mi, ni) for this lane,
// relative to the workgroup tile origin.
__device__ __forceinline__ int acc_m(int mi, int r) {
  const int lane = threadIdx.x & 63, wm = (threadIdx.x >> 6) >> 1;
  return wm * 128 + mi * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
}
__device__ __forceinline__ int acc_n(int ni) {
  const int lane = threadIdx.x & 63, wn = (threadIdx.x >> 6) & 1;
  return wn * 128 + ni * 32 + (lane & 31);
}

}  // namespace gemm
}  // namespace rbp
