// bf16 MFMA tile definitions for gfx950 (CDNA4), shared by the products of
// the log-prob path, all written as  C[m][n] = sum_k A(m, k) * B(n, k)  with
// fp32 accumulation:
//   logits   A = W  (m = vocabulary), B = H  (n = token), k = hidden unit
//   dhidden  A = W^T (m = hidden unit), B = dz (n = token), k = vocabulary
//   dW       A = H^T (m = hidden unit), B = dz^T (n = vocabulary), k = token
// Each operand is read where it lies, k-contiguous ("K-major") or
// m/n-contiguous ("MN-major"); one mainloop (gemm_dma.h) serves all of them.
//
// Workgroup tile 256 x 256 over a grid of WM x WN waves; each wave owns
// (256/WM) x (256/WN) outputs as MI x NI v_mfma_f32_32x32x16_bf16 tiles.
// MFMA 32x32x16 lane layout: lane l supplies A[l % 32][8 (l / 32) .. + 8) and
// B[l % 32][8 (l / 32) .. + 8); accumulator r of lane l holds
// C[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].  Each lane therefore owns runs of
// four consecutive m for one n (the fp32 epilogues store them as 16-byte
// vectors); with B loaded with paired rows it owns two adjacent n of the same
// m, which the bf16 epilogues store as one 4-byte pair.
//
// An LDS operand tile is [256 rows][64 k] bf16: 128-byte rows of eight 16-byte
// chunks, chunk index XOR-swizzled by (row ^ row >> 3) & 7 so that fragment
// reads (32 consecutive rows, one chunk) hit distinct banks whether the LDS
// serves 8 or 16 lanes of a 16-byte access per cycle.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace rbp {
namespace gemm {

typedef __bf16 bf16x8 __attribute__((__vector_size__(16)));
typedef float f32x16 __attribute__((__vector_size__(64)));

constexpr int kTileBytes = 256 * 64 * 2;   // one operand tile, 32 KiB
// five operand tiles -- three buffers of one operand, two of the other --
// 160 KiB, the whole LDS of a gfx950 compute unit (gemm_dma.h)
constexpr int kLdsBytes = 5 * kTileBytes;

// Stored operand: element (mn, k) is ptr[mn * ld + k].  Reads outside
// [0, mn_extent) x [0, k_extent) are replaced by zeros; k_extent % 8 == 0
// (16-byte vectors never straddle the edge).
struct Operand {
  const uint16_t* ptr;
  int64_t ld;
  int64_t mn_extent;
  int64_t k_extent;
};

// Byte offset beyond every buffer resource built here: loads there read zero.
constexpr uint32_t kOutOfRange = 0x7ffffff0u;

// Scheduling fence: the compiler may not move instructions across it, which
// keeps fragment reads issued one K slice ahead of the MFMAs that use them.
#define RBP_FENCE() __builtin_amdgcn_sched_barrier(0)

// Wave grid: WM x WN waves over the 256 x 256 tile.
template <int WM_, int WN_>
struct Grid {
  static constexpr int WM = WM_, WN = WN_;
  static constexpr int kWaves = WM * WN;
  static constexpr int kThreads = 64 * kWaves;
  static constexpr int MI = 256 / 32 / WM;
  static constexpr int NI = 256 / 32 / WN;
  static __device__ __forceinline__ int wave() { return threadIdx.x >> 6; }
  static __device__ __forceinline__ int wm() { return wave() / WN; }
  static __device__ __forceinline__ int wn() { return wave() % WN; }
  // row (m) / column (n) of accumulator r of MFMA tile (mi, ni), tile-relative
  static __device__ __forceinline__ int row(int mi, int r) {
    return wm() * (256 / WM) + mi * 32 + (r >> 2) * 8 + ((threadIdx.x & 63) >> 5) * 4 + (r & 3);
  }
  // row(mi, r) - row(0, 0): a compile-time constant for unrolled mi, r
  static __device__ __forceinline__ constexpr int row_off(int mi, int r) {
    return mi * 32 + (r >> 2) * 8 + (r & 3);
  }
  static __device__ __forceinline__ int col(int ni) {
    return wn() * (256 / WN) + ni * 32 + (threadIdx.x & 31);
  }
  // column of tile ni when B is loaded with paired rows (gemm_dma.h,
  // kKPaired): lane l of tiles 0 and 1 holds columns 2 (l % 32) and
  // 2 (l % 32) + 1 of the wave's 64
  static __device__ __forceinline__ int col_paired(int ni) {
    static_assert(256 / WN == 64 && NI == 2, "paired columns need 64-column waves");
    return wn() * 64 + 2 * (threadIdx.x & 31) + ni;
  }
};
// 8 waves, two per SIMD, 128 x 64 outputs each (128 accumulators per lane):
// enough waves keep loads in flight to feed a 256 x 256 tile.
using Grid8 = Grid<2, 4>;

// Block id -> (tile_m, tile_n).  The dispatcher hands block b to XCD b % 8, so
// blocks are first renumbered XCD by XCD (each XCD gets a contiguous range of
// tiles), then rastered in groups of `group_m` M-tiles per N-tile: the ~32
// blocks an XCD runs at once form a compact group_m x (32 / group_m) patch
// whose operand rows are shared through that XCD's L2.
__device__ __forceinline__ void map_tile(int32_t bid, int32_t tiles_m, int32_t tiles_n,
                                         int32_t group_m, int32_t& tm, int32_t& tn) {
  const uint32_t nblk = (uint32_t)tiles_m * (uint32_t)tiles_n;
  const uint32_t xcd = (uint32_t)bid & 7u, local = (uint32_t)bid >> 3;
  const uint32_t per = nblk >> 3, rem = nblk & 7u;
  const uint32_t L = xcd < rem ? xcd * (per + 1) + local
                               : rem * (per + 1) + (xcd - rem) * per + local;
  const uint32_t group_size = (uint32_t)group_m * (uint32_t)tiles_n;
  const uint32_t g = L / group_size;
  const uint32_t first_m = g * (uint32_t)group_m;
  const uint32_t gm = ((uint32_t)tiles_m - first_m) < (uint32_t)group_m
                          ? ((uint32_t)tiles_m - first_m)
                          : (uint32_t)group_m;
  const uint32_t in = L - g * group_size;
  tm = (int32_t)(first_m + in % gm);
  tn = (int32_t)(in / gm);
}

}  // namespace gemm
}  // namespace rbp
