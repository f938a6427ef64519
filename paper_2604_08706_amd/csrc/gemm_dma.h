// The K loop of every bf16 product: operands streamed HBM -> LDS with direct
// loads (gfx950 buffer_load_dwordx4 ... lds), K step 64, one operand in three
// LDS buffers and the other in two (160 KiB, the whole LDS).
//
// * Direct loads need no staging registers and no ds_write instructions.  A
//   load instruction writes 64 lanes x 16 bytes to LDS at M0 + 16 * lane, i.e.
//   8 consecutive 128-byte rows; the bank swizzle (gemm_core.h) is applied on
//   the HBM side -- the lane that lands on physical chunk p of row `row`
//   fetches logical chunk p ^ swz(row).
// * 128-byte rows make every row segment a whole cache line: measured L2 ->
//   CU rate ~28 TB/s for 128-byte segments against ~16 TB/s for 64-byte ones.
// * Both operands' loads of step s + 2 are issued during step s, spread
//   between MFMAs so the wave's MFMA issue never waits behind a burst of
//   loads: the three-buffer ("deep") operand's in the first K slice, the
//   other's right after the barrier that frees its buffer, in the last.  A
//   fill therefore has ~1.75 (deep) or ~1 step of MFMAs to land, where two
//   buffers per operand gave ~1 and ~0.75: operand rows missing the L2 (every
//   step's first request for a panel row goes to the Infinity Cache or HBM)
//   arrive before the barrier that needs them.
// * Fragments are read one K slice (16) ahead of the MFMAs that use them; the
//   first slice of step s + 1 is read right after the barrier, while the last
//   slice of step s (already in registers) multiplies.
// * An operand is stored either K-major (k contiguous: tile = 256 rows of
//   128 bytes per K step) or MN-major (m contiguous: tile = 64 K rows of 512
//   bytes).  MN-major tiles are read with the gfx950 transpose load
//   (ds_read_b64_tr_b16), which regroups 16-bit elements across lanes so the
//   MFMA operand comes out k-contiguous per lane without any transpose pass.
// * The loads are issued with inline assembly and their completion is tracked
//   by hand (s_waitcnt vmcnt): the compiler's own tracking of LDS-DMA waits for
//   every outstanding load before each LDS read and would serialize the
//   pipeline.  Nothing else in these kernels touches M0 or issues vector memory
//   loads inside the loop, and the loop ends with vmcnt(0).
#pragma once

#include <type_traits>

#include "gemm_core.h"

namespace rbp {
namespace gemm {

constexpr int kBK = 64;

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource as four SGPRs: 48-bit base, stride 0, range in bytes.
__device__ __forceinline__ i32x4 rsrc_words(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)a, (int)((a >> 32) & 0xffffu), (int)bytes, 0x00020000};
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane from buffer offset `voff` into LDS at lds + 16 * lane.
__device__ __forceinline__ void dma16(uint32_t lds, uint32_t voff, i32x4 rsrc) {
  // the resource is wave-uniform; say so where the compiler cannot prove it
#pragma unroll
  for (int i = 0; i < 4; ++i) rsrc[i] = __builtin_amdgcn_readfirstlane(rsrc[i]);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// s_waitcnt encodings (gfx9): vmcnt in bits [3:0] and [15:14], expcnt [6:4],
// lgkmcnt [11:8]; other counters left at their maximum.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xf << 8));
}

// vmcnt(N) and lgkmcnt(0) in one wait.
template <int N>
__device__ __forceinline__ void wait_vmcnt_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4));
}

// Workgroup barrier that is also a compiler memory barrier: LDS reads after it
// may not be moved above it (s_barrier alone orders no memory accesses).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

template <class G>
__device__ __forceinline__ void mfma_tiles(const bf16x8 (&a)[G::MI], const bf16x8 (&b)[G::NI],
                                           f32x16 (&acc)[G::MI][G::NI]) {
#pragma unroll
  for (int mi = 0; mi < G::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < G::NI; ++ni)
      acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
}

// MFMAs of one K slice with `nload` loads spread evenly between them: a
// burst of loads would stall this wave's MFMA issue while the CU's address
// unit accepts them.  load(l) issues load l (or nothing).
template <class G, class LoadFn>
__device__ __forceinline__ void mfma_tiles_interleaved(const bf16x8 (&a)[G::MI],
                                                       const bf16x8 (&b)[G::NI],
                                                       f32x16 (&acc)[G::MI][G::NI], int nload,
                                                       LoadFn&& load) {
  constexpr int M = G::MI * G::NI;
  const int every = M / nload;
#pragma unroll
  for (int q = 0; q < M; ++q) {
    const int mi = q / G::NI, ni = q % G::NI;
    acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    if ((q + 1) % every == 0 && (q + 1) / every <= nload) {
      RBP_FENCE();
      load((q + 1) / every - 1);
      RBP_FENCE();
    }
  }
}

// Operand layouts (template arguments of tile_stream):
//   kKMajor   element (mn, k) at ptr[mn * ld + k];
//   kMNMajor  element (mn, k) at ptr[k * ld + mn];
//   kKPaired  K-major, with the rows of every 64-row block reordered on their
//             way into LDS: rows 2 i and 2 i + 1 land in LDS rows i and 32 + i,
//             so the two 32-row MFMA tiles of a 64-row wave block hold the
//             block's even and odd rows, and one lane holds the outputs of two
//             adjacent rows (Grid::col_paired).
constexpr int kKMajor = 0, kMNMajor = 1, kKPaired = 2;

// ---- K-major operand: LDS tile = 256 rows x 128 bytes (K step 64) ----------
//
// Each lane's share of one operand tile's loads.  Load j of a wave moves a
// 1 KiB block (8 rows x 128 bytes) into LDS; the offsets are relative to the
// first row of the tile, so they serve every tile of a launch.  With kPaired
// LDS row r holds operand row (r & ~63) | 2 (r & 31) | ((r >> 5) & 1); the
// swizzle follows the LDS row.
template <class G, bool kPaired>
struct KLanes {
  static constexpr int kLoads = 32 / G::kWaves;  // 1 KiB blocks per wave per step
  uint32_t voff[kLoads];
  int kc[kLoads];

  __device__ __forceinline__ void init(int64_t ld) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // block b = j * kWaves + wave holds rows 8 b .. 8 b + 7; lane -> row
    // 8 b + lane / 8, physical chunk lane % 8, logical chunk
    // (lane % 8) ^ swz(row), swz(row) = (row ^ (row >> 3)) & 7 = (lane / 8) ^ (b & 7)
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int b = j * G::kWaves + wave;
      const int row = b * 8 + (lane >> 3);
      const int src = kPaired ? ((row & ~63) | ((row & 31) << 1) | ((row >> 5) & 1)) : row;
      const int c = (lane & 7) ^ (lane >> 3) ^ (b & 7);
      kc[j] = c * 8;
      voff[j] = (uint32_t)((src * ld + c * 8) * 2);
    }
  }
};

// Buffer resource over the (at most 256) rows of `op` starting at mn0: rows
// past the operand's end read as zero.
__device__ __forceinline__ i32x4 tile_rsrc(const Operand& op, int64_t mn0) {
  int64_t rows = op.mn_extent - mn0;
  rows = rows < 0 ? 0 : (rows > 256 ? 256 : rows);
  return rsrc_words(op.ptr + mn0 * op.ld, (uint32_t)(rows * op.ld * 2));
}

// Fragment reads from a K-major tile (gemm_core.h swizzle): slice ks, row
// block i reads base[((2 ks) ^ (4 (i & 1))) / 2] + 4096 i.
template <int kCount>
struct KFrags {
  uint32_t base[4];
  __device__ __forceinline__ void init(uint32_t tile_off, int wave_rows) {
    const int lane = threadIdx.x & 63;
    const int r = lane & 31;
    const int t = (lane >> 5) ^ (r & 7) ^ (r >> 3);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      base[j] = tile_off + (uint32_t)(wave_rows * 128 + r * 128 + (((2 * j) ^ t) << 4));
  }
  __device__ __forceinline__ void read(const uint8_t* stage, int ks, bf16x8 (&v)[kCount]) const {
#pragma unroll
    for (int i = 0; i < kCount; ++i)
      v[i] = *reinterpret_cast<const bf16x8*>(stage + base[((2 * ks) ^ (4 * (i & 1))) >> 1] +
                                              4096 * i);
  }
};

// ---- MN-major operand: LDS tile = 64 K rows x 512 bytes ---------------------
//
// Row r of the tile (K index k0 + r) holds the tile's 256 m as 32 chunks of
// 16 bytes; logical chunk c sits at physical chunk c ^ (4 (r & 3)), i.e. the
// four 64-byte quarters of each 256-byte half are rotated by row, so the
// 8-byte transpose reads of one half-wave (4 K rows x 64 bytes) cover all
// banks once.  Load j of a wave moves 2 rows (1 KiB); a lane fetches logical
// chunk c ^ (4 (r & 3)) for physical chunk c = lane % 32.
template <class G>
struct MNLanes {
  static constexpr int kLoads = 32 / G::kWaves;
  uint32_t voff[kLoads];  // relative to element (k0, m0) of the step
  int col[kLoads];        // first m of the chunk, relative to m0

  __device__ __forceinline__ void init(int64_t ld) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int b = j * G::kWaves + wave;
      const int r = 2 * b + (lane >> 5);
      const int c = (lane & 31) ^ ((r & 3) << 2);
      col[j] = c * 8;
      voff[j] = (uint32_t)((r * ld + c * 8) * 2);
    }
  }
};

// gfx950 transpose load: lane 16 g + i receives, as element e (0..3), the
// 16-bit value at byte 2 (i % 4) of the 8 bytes addressed by lane
// 16 g + 4 e + i / 4.
__device__ __forceinline__ uint64_t lds_read_tr16(const uint8_t* p) {
  typedef __bf16 bf16x4 __attribute__((__vector_size__(8)));
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  const auto* q = reinterpret_cast<const __attribute__((address_space(3))) uint8_t*>(
      (uint32_t)reinterpret_cast<uintptr_t>(p));
  const bf16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)q);
  return __builtin_bit_cast(uint64_t, v);
}

// Fragment reads from an MN-major tile.  The MFMA operand wants lane l to hold
// X[m = l % 32][k = 8 (l / 32) .. + 8]; by the transpose-load rule above, lane
// s must address K row kr = 8 (s / 32) + 4 h + (s % 16) / 4 (h = which half of
// the 8 k) at m = 16 ((s / 16) % 2) + 4 (s % 4) within the 32-m block.
template <int kCount>
struct MNFrags {
  uint32_t base[kCount];
  __device__ __forceinline__ void init(uint32_t tile_off, int wave_rows) {
    const int s = threadIdx.x & 63;
    const int q = (s & 15) >> 2;  // == kr & 3
    const int kr = 8 * (s >> 5) + q;
    const int mb = 2 * (16 * ((s >> 4) & 1) + 4 * (s & 3));  // byte within a 64-byte block
#pragma unroll
    for (int i = 0; i < kCount; ++i)
      base[i] = tile_off + (uint32_t)(kr * 512 + mb + ((2 * wave_rows + 64 * i) ^ (64 * q)));
  }
  __device__ __forceinline__ void read(const uint8_t* stage, int ks, bf16x8 (&v)[kCount]) const {
#pragma unroll
    for (int i = 0; i < kCount; ++i) {
      const uint8_t* p = stage + base[i] + ks * (16 * 512);
      const uint64_t lo = lds_read_tr16(p), hi = lds_read_tr16(p + 4 * 512);
      typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));
      v[i] = __builtin_bit_cast(bf16x8, u64x2{lo, hi});
    }
  }
};

template <int kLayout, int kCount>
using Frags =
    typename std::conditional<kLayout == kMNMajor, MNFrags<kCount>, KFrags<kCount>>::type;

// One output tile: rows m0.. of A, rows n0.. of B, K range [k_begin, k_end)
// (non-empty).  32-bit fields keep the loop's scalar state small.
struct Tile {
  int32_t m0, n0, k_begin, k_end;
};

__device__ __forceinline__ int32_t k_steps(const Tile& t) {
  return (t.k_end - t.k_begin + kBK - 1) / kBK;
}

// Load side of one operand: per-lane offsets, the per-tile view (`Res`) and
// the issue of load j of K step `step` of a tile into an LDS tile.
template <class G, int kLayout>
struct SideLoad {  // K-major (kKMajor, kKPaired)
  KLanes<G, kLayout == kKPaired> lanes;
  int32_t k_extent;
  struct Res {
    i32x4 rsrc;  // the tile's (at most 256) rows; range 0 past the end of the stream
    int32_t kb;  // first K column of the tile
  };
  __device__ __forceinline__ void init(const Operand& op) {
    lanes.init(op.ld);
    k_extent = (int32_t)op.k_extent;
  }
  __device__ __forceinline__ Res res(const Operand& op, int32_t mn0, int32_t kb,
                                     bool valid) const {
    Res r;
    r.rsrc = valid ? tile_rsrc(op, mn0) : rsrc_words(op.ptr, 0u);
    r.kb = kb;
    return r;
  }
  __device__ __forceinline__ void issue(uint32_t tile, const Res& r, int32_t step, int j) const {
    const uint32_t wave = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int32_t k0 = r.kb + step * kBK;
    const bool ok = k0 + lanes.kc[j] < k_extent;  // columns past K read zero
    dma16(tile + (uint32_t)(j * G::kWaves + wave) * 1024u,
          ok ? lanes.voff[j] + (uint32_t)(k0 * 2) : kOutOfRange, r.rsrc);
  }
};

template <class G>
struct SideLoad<G, kMNMajor> {
  MNLanes<G> lanes;
  int32_t mn_extent;
  int64_t ld;
  struct Res {
    uint64_t addr;  // byte address of element (k = kb, mn0)
    int32_t krem;   // K rows left from kb (0 past the end of the stream)
    int32_t mn0;
  };
  int32_t k_extent;
  __device__ __forceinline__ void init(const Operand& op) {
    lanes.init(op.ld);
    mn_extent = (int32_t)op.mn_extent;
    k_extent = (int32_t)op.k_extent;
    ld = op.ld;
  }
  __device__ __forceinline__ Res res(const Operand& op, int32_t mn0, int32_t kb,
                                     bool valid) const {
    Res r;
    r.addr = reinterpret_cast<uint64_t>(op.ptr + (int64_t)kb * op.ld + mn0);
    r.krem = valid ? k_extent - kb : 0;
    r.mn0 = mn0;
    return r;
  }
  __device__ __forceinline__ void issue(uint32_t tile, const Res& r, int32_t step, int j) const {
    const uint32_t wave = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // this step's K rows as one resource: rows past K read zero
    int32_t rows = r.krem - step * kBK;
    rows = rows < 0 ? 0 : (rows > kBK ? kBK : rows);
    const i32x4 rsrc =
        rsrc_words(reinterpret_cast<const void*>(r.addr + (uint64_t)step * kBK * ld * 2),
                   (uint32_t)(rows * ld * 2));
    const bool ok = r.mn0 + lanes.col[j] < mn_extent;  // m past the operand reads zero
    dma16(tile + (uint32_t)(j * G::kWaves + wave) * 1024u, ok ? lanes.voff[j] : kOutOfRange,
          rsrc);
  }
};

// Persistent tile loop.  This workgroup takes the virtual blocks blockIdx.x,
// blockIdx.x + gridDim.x, ... below n_vid; tile_of(vid) gives each one's Tile
// (every tile of a launch has the same number of K steps, nk >= 1) and
// epi(vid, acc) consumes its finished fp32 accumulators.  An epi that
// returns bool may return false to keep the accumulators for the
// workgroup's next virtual block (whose K range then continues the same
// output tile); one that returns void always starts the next block from
// zero.  kLA / kLB select the layouts of A / B (kKMajor, kMNMajor,
// kKPaired); K-major needs k_extent % 8 == 0, MN-major mn_extent % 8 == 0.
// kDeep names the operand with three buffers (1: A, 2: B); smem holds
// kLdsBytes: the deep operand's buffers, then the other's two.
//
// The K steps of consecutive tiles form one stream through the buffers (step
// g of the stream in deep buffer g % 3 and other buffer g % 2), so the first
// steps of the next tile load while the current tile's last steps multiply
// and its epilogue runs.  Per step g, with slice 0's fragments already in
// registers:
//   slice 0: read slice 1; MFMAs; issue the deep operand's loads of step
//            g + 2 into its buffer (g + 2) % 3 (free since the barrier of
//            step g - 1);
//   slices 1, 2: read the next slice; MFMAs;
//   wait until only those loads are outstanding (step g + 1 landed) and for
//   this wave's LDS reads; barrier (step g + 1 visible to all; step g's
//   buffers no longer read);
//   slice 3: read step g + 1's slice 0; MFMAs; issue the other operand's
//            loads of step g + 2 into its buffer g % 2;
//   after the last step of a tile: epi(), which may not use LDS (every byte
//   of it is a buffer) and may contain barriers.
// The load cursor runs two steps ahead of the MFMAs and recomputes its view
// whenever it enters a new tile.
template <class G, int kLA, int kLB, int kDeep, class TileFn, class EpiFn>
__device__ __forceinline__ void tile_stream(const Operand& A, const Operand& B, int32_t n_vid,
                                            uint8_t* smem, TileFn&& tile_of, EpiFn&& epi) {
  static_assert(kDeep == 1 || kDeep == 2, "deep operand: 1 = A, 2 = B");
  constexpr int nA = kDeep == 1 ? 3 : 2;
  const int32_t stride = (int32_t)gridDim.x;
  const int32_t vid0 = (int32_t)blockIdx.x;
  if (vid0 >= n_vid) return;
  constexpr int L = 32 / G::kWaves;
  SideLoad<G, kLA> la;
  SideLoad<G, kLB> lb;
  la.init(A);
  lb.init(B);
  Frags<kLA, G::MI> fa;
  Frags<kLB, G::NI> fb;
  fa.init(0u, G::wm() * (256 / G::WM));
  fb.init(0u, G::wn() * (256 / G::WN));
  const uint32_t ldsA = (uint32_t)reinterpret_cast<uintptr_t>(smem);
  const uint32_t ldsB = ldsA + (uint32_t)(nA * kTileBytes);
  const uint8_t* smA = smem;
  const uint8_t* smB = smem + nA * kTileBytes;
  const int32_t nk = k_steps(tile_of(vid0));

  struct TileRes {
    typename SideLoad<G, kLA>::Res a;
    typename SideLoad<G, kLB>::Res b;
  };
  auto res_of = [&](int32_t vid) {
    const bool valid = vid < n_vid;
    const Tile t = tile_of(valid ? vid : vid0);
    return TileRes{la.res(A, t.m0, t.k_begin, valid), lb.res(B, t.n0, t.k_begin, valid)};
  };
  // load cursor: tile qvid (view cur), K step qs
  int32_t qvid = vid0, qs = 0;
  TileRes cur = res_of(vid0);
  auto advance = [&]() {
    if (++qs == nk) {
      qs = 0;
      qvid += stride;
      cur = res_of(qvid);
    }
  };
  auto issue_a = [&](uint32_t buf, int j) {
    la.issue(ldsA + buf * (uint32_t)kTileBytes, cur.a, qs, j);
  };
  auto issue_b = [&](uint32_t buf, int j) {
    lb.issue(ldsB + buf * (uint32_t)kTileBytes, cur.b, qs, j);
  };
  auto read = [&](uint32_t ba, uint32_t bb, int ks, bf16x8 (&a)[G::MI], bf16x8 (&b)[G::NI]) {
    fa.read(smA + ba * kTileBytes, ks, a);
    fb.read(smB + bb * kTileBytes, ks, b);
  };
  // buffers of the deep operand for steps g, g + 1, g + 2 (rotating mod 3)
  // and of the other for step g (its step g + 1 is the other buffer, and its
  // step g + 2 reuses step g's)
  uint32_t d0 = 0, d1 = 1, d2 = 2, o0 = 0;

  // prologue: steps 0 and 1 issued, step 0 landed, cursor at step 2
#pragma unroll
  for (int j = 0; j < L; ++j) issue_a(0u, j);
#pragma unroll
  for (int j = 0; j < L; ++j) issue_b(0u, j);
  advance();
#pragma unroll
  for (int j = 0; j < L; ++j) issue_a(1u, j);
#pragma unroll
  for (int j = 0; j < L; ++j) issue_b(1u, j);
  advance();
  wait_vmcnt<2 * L>();
  lds_barrier();

  int32_t mvid = vid0, mit = 0;
  f32x16 acc[G::MI][G::NI];
#pragma unroll
  for (int mi = 0; mi < G::MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < G::NI; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;
  bf16x8 a0[G::MI], b0[G::NI], a1[G::MI], b1[G::NI];
  read(0u, 0u, 0, a0, b0);
  for (;;) {
    const uint32_t ca = kDeep == 1 ? d0 : o0, cb = kDeep == 2 ? d0 : o0;
    const uint32_t na = kDeep == 1 ? d1 : (o0 ^ 1u), nb = kDeep == 2 ? d1 : (o0 ^ 1u);
    read(ca, cb, 1, a1, b1);
    RBP_FENCE();
    mfma_tiles_interleaved<G>(a0, b0, acc, L, [&](int l) {
      if constexpr (kDeep == 1)
        issue_a(d2, l);
      else
        issue_b(d2, l);
    });
    RBP_FENCE();
    read(ca, cb, 2, a0, b0);
    RBP_FENCE();
    mfma_tiles<G>(a1, b1, acc);
    RBP_FENCE();
    read(ca, cb, 3, a1, b1);
    RBP_FENCE();
    mfma_tiles<G>(a0, b0, acc);
    RBP_FENCE();
    // step g + 1 landed (only the deep operand's step g + 2 loads are
    // outstanding); this wave's reads of step g done
    wait_vmcnt_lgkm0<L>();
    lds_barrier();
    // unconditional (after the last step it reads a stale buffer)
    read(na, nb, 0, a0, b0);
    RBP_FENCE();
    mfma_tiles_interleaved<G>(a1, b1, acc, L, [&](int l) {
      if constexpr (kDeep == 1)
        issue_b(o0, l);
      else
        issue_a(o0, l);
    });
    RBP_FENCE();
    advance();
    {
      const uint32_t t = d0;
      d0 = d1;
      d1 = d2;
      d2 = t;
      o0 ^= 1u;
    }
    if (++mit == nk) {
      bool done = true;
      if constexpr (std::is_same_v<decltype(epi(mvid, acc)), bool>)
        done = epi(mvid, acc);
      else
        epi(mvid, acc);
      if (done) {
#pragma unroll
        for (int mi = 0; mi < G::MI; ++mi)
#pragma unroll
          for (int ni = 0; ni < G::NI; ++ni)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[mi][ni][r] = 0.0f;
      }
      mvid += stride;
      if (mvid >= n_vid) break;
      mit = 0;
    }
  }
  wait_vmcnt<0>();
}

// Workgroups for a persistent launch over n_tiles tiles on a device with
// n_cu compute units (one 256 x 256 workgroup per CU): a multiple of 8, so a
// virtual block keeps the XCD (block id mod 8) of the workgroup that runs it.
inline int64_t stream_grid(int64_t n_tiles, int n_cu) {
  int64_t g = n_cu < 8 ? 8 : (n_cu / 8) * 8;
  const int64_t need = (n_tiles + 7) / 8 * 8;
  return g < need ? g : need;
}

}  // namespace gemm
}  // namespace rbp
