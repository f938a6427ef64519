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
constexpr int kTileBytes = 256 * kBK * 2;  // one operand tile, 32 KiB
constexpr int kLdsBytes = 4 * kTileBytes;  // A stage 0, A stage 1, B stage 0, B stage 1
constexpr int kOffA0 = 0, kOffA1 = kTileBytes, kOffB0 = 2 * kTileBytes, kOffB1 = 3 * kTileBytes;

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

// Byte offset that lies outside every buffer resource built below: a load
// there returns zeros.
constexpr uint32_t kOutOfRange = 0x7ffffff0u;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  // raw (stride 0) buffer; loads at byte offsets >= `bytes` read as zero
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// Loader of one 256 x 64 operand tile per K step, HBM -> registers, through
// buffer loads whose range check zero-fills every tail.
template <bool KMAJOR>
struct TileLoader;

// Element (mn, k) at ptr[mn * ld + k].  Thread -> rows tid/8 + 32 p, chunk
// tid % 8: 8 lanes read one 128-byte run of a row.  One resource covers the
// tile's valid rows; the K tail is zero-filled per thread.
template <>
struct TileLoader<true> {
  __amdgpu_buffer_rsrc_t rsrc;
  uint32_t voff[8];
  int64_t k_extent;
  int k_thread;

  __device__ __forceinline__ void init(const Operand& op, int64_t mn0) {
    const int tid = threadIdx.x;
    int64_t rows = op.mn_extent - mn0;
    rows = rows < 0 ? 0 : (rows > 256 ? 256 : rows);
    rsrc = make_rsrc(op.ptr + mn0 * op.ld, (uint32_t)(rows * op.ld * 2));
#pragma unroll
    for (int p = 0; p < 8; ++p)
      voff[p] = (uint32_t)((((tid >> 3) + 32 * p) * op.ld + (tid & 7) * 8) * 2);
    k_extent = op.k_extent;
    k_thread = (tid & 7) * 8;
  }
  __device__ __forceinline__ void load(int64_t k0, u32x4 (&r)[8]) const {
    const bool ok = k0 + k_thread < k_extent;
    const uint32_t kb = (uint32_t)(k0 * 2);
#pragma unroll
    for (int p = 0; p < 8; ++p)
      r[p] = __builtin_amdgcn_raw_buffer_load_b128(rsrc, ok ? voff[p] + kb : kOutOfRange, 0, 0);
  }
};

// Element (mn, k) at ptr[k * ld + mn].  Thread -> 8 x 8 block (k rows
// kb*8.., mn columns mb*8..); 32 lanes read 512 contiguous bytes of one k row.
// The resource is rebuilt per K step at that step's first row, so offsets stay
// small and rows past the K extent read as zero; the MN tail is zero-filled
// per thread.
template <>
struct TileLoader<false> {
  const uint16_t* base;
  int64_t ld, k_extent;
  uint32_t voff[8];
  bool mn_ok;

  __device__ __forceinline__ void init(const Operand& op, int64_t mn0) {
    const int tid = threadIdx.x;
    const int kb = tid >> 5, mb = tid & 31;
    base = op.ptr + mn0;
    ld = op.ld;
    k_extent = op.k_extent;
    mn_ok = mn0 + mb * 8 < op.mn_extent;
#pragma unroll
    for (int q = 0; q < 8; ++q) voff[q] = (uint32_t)(((kb * 8 + q) * op.ld + mb * 8) * 2);
  }
  __device__ __forceinline__ void load(int64_t k0, u32x4 (&r)[8]) const {
    int64_t rows = k_extent - k0;
    rows = rows < 0 ? 0 : (rows > 64 ? 64 : rows);
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(base + k0 * ld, (uint32_t)(rows * ld * 2));
#pragma unroll
    for (int q = 0; q < 8; ++q)
      r[q] = __builtin_amdgcn_raw_buffer_load_b128(rs, mn_ok ? voff[q] : kOutOfRange, 0, 0);
  }
};

// Registers -> LDS tile (transposing MN-major blocks).
//
// Address algebra of the swizzle lds_off(row, chunk) = row*128 +
// ((chunk ^ row ^ (row >> 3)) & 7)*16, used to keep every LDS address a
// per-lane base plus a compile-time immediate:
//  * K-major store, row = tid/8 + 32p: (row >> 3) & 7 = (tid >> 6) ^ 4(p & 1),
//    so the address is base[p & 1] + 4096 p;
//  * fragment read, row = R0 + 32i + r (R0 a multiple of 128, r = lane % 32),
//    chunk = 2ks + lane/32: the physical chunk is (2ks ^ 4(i & 1)) ^ t with a
//    per-lane t, so the address is frag[(2ks ^ 4(i & 1)) / 2] + 4096 i.
template <bool KMAJOR>
__device__ __forceinline__ void store_tile(const u32x4 (&r)[8], uint8_t* tile) {
  const int tid = threadIdx.x;
  if constexpr (KMAJOR) {
    const int chunk = tid & 7, row0 = tid >> 3;
    const int u = chunk ^ (row0 & 7) ^ (tid >> 6);
    uint8_t* const b0 = tile + row0 * 128 + (u << 4);
    uint8_t* const b1 = tile + row0 * 128 + ((u ^ 4) << 4);
#pragma unroll
    for (int p = 0; p < 8; ++p)
      *reinterpret_cast<u32x4*>(((p & 1) ? b1 : b0) + 4096 * p) = r[p];
  } else {
    const int kb = tid >> 5, mb = tid & 31;
    const int v = kb ^ (mb & 7);
    uint8_t* const b = tile + mb * 1024;
    // r[q] holds k row q, bf16 columns c = 0..7 (column c in dword c/2, half c%2).
    // Output row c gets, in dword q, (k = 2q, k = 2q + 1) of column c.
#pragma unroll
    for (int c = 0; c < 8; ++c) {
      const uint32_t sel = (c & 1) ? 0x07060302u : 0x05040100u;
      u32x4 o;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        o[q] = __builtin_amdgcn_perm(r[2 * q + 1][c >> 1], r[2 * q][c >> 1], sel);
      *reinterpret_cast<u32x4*>(b + c * 128 + ((v ^ c) << 4)) = o;
    }
  }
}

// Per-lane fragment read bases (byte offsets within an operand tile, for the
// wave's row block R0): frag[j] serves physical chunk pattern 2j.
struct FragBase {
  int a[4], b[4];
};

__device__ __forceinline__ FragBase frag_bases() {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int r = lane & 31;
  const int t = (lane >> 5) ^ (r & 7) ^ (r >> 3);  // (row >> 3) & 7 = r >> 3 for i = 0
  FragBase f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int off = r * 128 + (((2 * j) ^ t) << 4);
    f.a[j] = wm * 128 * 128 + off;
    f.b[j] = wn * 128 * 128 + off;
  }
  return f;
}

// Fragments of K slice ks (16 wide) for this wave: 4 A and 4 B row blocks.
__device__ __forceinline__ void load_frags(const uint8_t* tA, const uint8_t* tB,
                                           const FragBase& f, int ks, bf16x8 (&a)[4],
                                           bf16x8 (&b)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = ((2 * ks) ^ (4 * (i & 1))) >> 1;
    a[i] = *reinterpret_cast<const bf16x8*>(tA + f.a[j] + 4096 * i);
    b[i] = *reinterpret_cast<const bf16x8*>(tB + f.b[j] + 4096 * i);
  }
}

__device__ __forceinline__ void mfma_block(const bf16x8 (&a)[4], const bf16x8 (&b)[4],
                                           f32x16 (&acc)[4][4]) {
#pragma unroll
  for (int mi = 0; mi < 4; ++mi)
#pragma unroll
    for (int ni = 0; ni < 4; ++ni)
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
}

// Scheduling fence: the compiler may not move instructions across it, which
// keeps fragment reads issued one K slice ahead of the MFMAs that use them.
#define RBP_FENCE() __builtin_amdgcn_sched_barrier(0)

// Full K loop over [k_begin, k_end) for the tile at (m0, n0).
//
// Per step s (LDS stage s % 2 holds its operands):
//   issue the HBM loads of step s + 1 into registers;
//   for each K slice: read the next slice's fragments, then run this slice's
//     16 MFMAs (fenced, so LDS latency hides under 512 MFMA cycles);
//   before the last slice: write step s + 1 into the other LDS stage, barrier,
//     read step s + 1's first fragments -- the barrier and that read overlap
//     the last slice's MFMAs, whose operands are already in registers.
// Ends with a barrier, so the caller may reuse `smem` right away.
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
  TileLoader<A_KMAJOR> la;
  TileLoader<B_KMAJOR> lb;
  la.init(A, m0);
  lb.init(B, n0);
  const FragBase f = frag_bases();
  u32x4 ra[8], rb[8];
  bf16x8 a0[4], b0[4], a1[4], b1[4];
  la.load(k_begin, ra);
  lb.load(k_begin, rb);
  store_tile<A_KMAJOR>(ra, smem + kOffA0);
  store_tile<B_KMAJOR>(rb, smem + kOffB0);
  __syncthreads();
  load_frags(smem + kOffA0, smem + kOffB0, f, 0, a0, b0);
  for (int64_t it = 0; it < nk; ++it) {
    const int cur = (int)(it & 1);
    const uint8_t* tA = smem + (cur ? kOffA1 : kOffA0);
    const uint8_t* tB = smem + (cur ? kOffB1 : kOffB0);
    uint8_t* nA = smem + (cur ? kOffA0 : kOffA1);
    uint8_t* nB = smem + (cur ? kOffB0 : kOffB1);
    const bool more = it + 1 < nk;
    if (more) {
      la.load(k_begin + (it + 1) * kBK, ra);
      lb.load(k_begin + (it + 1) * kBK, rb);
    }
    RBP_FENCE();
    load_frags(tA, tB, f, 1, a1, b1);
    RBP_FENCE();
    mfma_block(a0, b0, acc);
    RBP_FENCE();
    load_frags(tA, tB, f, 2, a0, b0);
    RBP_FENCE();
    mfma_block(a1, b1, acc);
    RBP_FENCE();
    load_frags(tA, tB, f, 3, a1, b1);
    RBP_FENCE();
    mfma_block(a0, b0, acc);
    RBP_FENCE();
    if (more) {
      store_tile<A_KMAJOR>(ra, nA);
      store_tile<B_KMAJOR>(rb, nB);
    }
    __syncthreads();
    if (more) load_frags(nA, nB, f, 0, a0, b0);
    RBP_FENCE();
    mfma_block(a1, b1, acc);
    RBP_FENCE();
  }
  __syncthreads();
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
